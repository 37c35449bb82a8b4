// C ABI of libe2f (declared in include/e2f.h): argument checks on the host,
// the context with its coefficient tables and workspace, and the order of
// kernel launches for each entry point.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <algorithm>
#include <cstring>
#include <limits>
#include <map>
#include <string>
#include <vector>

#include "../../include/e2f.h"

#include "e2f_internal.h"
#include "e2f_launch.h"

using namespace e2f;

// Scratch memory of e2f_wigner6j_conv_forward_noalloc (for callers that
// cannot allocate): a file-scope device array, one copy per GPU, held until
// the process ends.  Host code never uses its name as an address: e2f_create
// resolves this device's copy with hipGetSymbolAddress and keeps the pointer.
constexpr size_t kScratchBytes = (size_t)128 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

thread_local std::string g_err;

e2f_status fail(e2f_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

struct Buf {
  void* p = nullptr;
  size_t n = 0;
};

}  // namespace

struct e2f_ctx {
  int device = -1;
  int lmax_max = 0;
  std::vector<LayerTables> host;
  std::vector<DevTables> dev;
  std::vector<void*> table_mem;            // structure arrays per L
  // path-weighted coefficients, one set per path-weight vector (per L, most
  // recently added last; at most kMaxCoefSets per L)
  struct CoefSet {
    std::vector<double> w;
    void* mem = nullptr;
    const double* q_coef = nullptr;
    const float* k_coef = nullptr;
    const double* rc_coef = nullptr;
    std::vector<const double*> rcf_coef;  // per filter degree f
    const float* w_f = nullptr;
    // fused recouple tensor (L <= kFuseMaxL): CSR over the positions of F
    // in the layout of nkr K rows
    struct FuseTab {
      const int* ptr = nullptr;
      const int* idx = nullptr;
      const double* coef = nullptr;
      int nkr = 0;
    };
    FuseTab f;
    // the passes of alpha / D^f (ynorm_passes), their degrees stacked in the
    // K rows
    std::vector<FuseTab> fy;
  };
  std::vector<std::vector<CoefSet>> coefs;
  // per L and filter degree f: the recouple schedule restricted to b + u = f
  std::vector<std::vector<const int*>> rcf_k, rcf_off, rcf_meta;
  int* stats = nullptr;                    // device, kStatsInts ints
  void* scratch = nullptr;                 // this device's copy of the file-scope scratch array
  int64_t* pinned = nullptr;               // host, 16 int64
  int32_t* pinned_plan = nullptr;          // host, plan sizes read back in one copy
  size_t pinned_plan_n = 0;
  Buf a, b, c;
  Buf d;                                   // backward staging (transposed graph, input gradient)
  std::vector<std::vector<double>> kappa;  // per L: [a][f][o] real CG transpose factors (0 = not computed)
  int64_t last_slices = 0;                 // receiver slices of the last factorised forward
  // kernel timing (e2f_profile): events recorded on the launch stream
  bool prof = false;
  struct Rec {
    const char* name;
    hipEvent_t start, stop;
  };
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
  // a second stream of the context's device and the events that fork work
  // onto it and join it back (the forward re-lays the features there while
  // the plan runs on the caller's stream)
  hipStream_t side = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  // coupling schedules of the aggregation of uncoupled products, per (L, groups)
  struct Couple {
    int k = 0, ntab = 0;
    int* meta = nullptr;
    float* coef = nullptr;
    int* pmeta = nullptr;  // packed entries and their coefficient table (ntab > 0)
    float* tab = nullptr;
  };
  std::map<std::pair<int, int>, Couple> couple;
  // schedules of the backward's filter contraction, per (L, rows per pass)
  struct Geom {
    int qc = 0, tot = 0;  // filter rows per pass, schedule entries
    int* meta = nullptr;
    float* unit = nullptr;
    int* oc = nullptr;  // [nchunk][2]: offset, steps
  };
  std::map<std::pair<int, int>, Geom> geom;  // per (L, head width)
};

namespace {

struct DeviceGuard {
  int prev = -1;
  bool ok = false;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    ok = hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceGuard() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

#define E2F_HIP(call)                                                                        \
  do {                                                                                       \
    hipError_t e_ = (call);                                                                  \
    if (e_ != hipSuccess) return fail(E2F_EDEVICE, "%s: %s", #call, hipGetErrorString(e_));  \
  } while (0)

size_t al256(size_t x) { return (x + 255) & ~size_t(255); }

hipEvent_t take_event(e2f_ctx* ctx) {
  if (!ctx->pool.empty()) {
    hipEvent_t e = ctx->pool.back();
    ctx->pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Brackets the launches of one named step with events when profiling is on.
struct Timed {
  e2f_ctx* ctx;
  hipStream_t s;
  e2f_ctx::Rec rec{};
  Timed(e2f_ctx* c, const char* name, hipStream_t st) : ctx(c), s(st) {
    if (!ctx->prof) return;
    rec.name = name;
    rec.start = take_event(ctx);
    rec.stop = take_event(ctx);
    if (rec.start) (void)hipEventRecord(rec.start, s);
  }
  ~Timed() {
    if (!ctx->prof || !rec.start || !rec.stop) return;
    (void)hipEventRecord(rec.stop, s);
    ctx->recs.push_back(rec);
  }
};

#define E2F_TIMED(name, call)            \
  do {                                   \
    Timed tm_(ctx, name, s);             \
    E2F_HIP(call);                       \
  } while (0)

e2f_status ensure(e2f_ctx* ctx, Buf& b, size_t bytes, hipStream_t s) {
  if (bytes <= b.n) return E2F_OK;
  if (b.p) {
    E2F_HIP(hipStreamSynchronize(s));
    E2F_HIP(hipFree(b.p));
    b.p = nullptr;
    b.n = 0;
  }
  size_t want = al256(bytes + bytes / 8);
  if (hipMalloc(&b.p, want) != hipSuccess) {
    (void)hipGetLastError();
    b.p = nullptr;
    return fail(E2F_ENOMEM, "workspace allocation of %zu bytes failed", want);
  }
  b.n = want;
  (void)ctx;
  return E2F_OK;
}

// Carves aligned sub-buffers out of one workspace.
struct Carver {
  char* base;
  size_t off = 0;
  template <typename T>
  T* take(size_t count) {
    T* p = (T*)(base + off);
    off += al256(sizeof(T) * count);
    return p;
  }
};

template <typename T>
void push_array(std::vector<char>& blob, std::vector<size_t>& offs, const std::vector<T>& v) {
  size_t off = al256(blob.size());
  blob.resize(off + sizeof(T) * std::max<size_t>(v.size(), 1), 0);
  if (!v.empty()) std::memcpy(blob.data() + off, v.data(), sizeof(T) * v.size());
  offs.push_back(off);
}

// The coupling schedule for (L, groups), uploaded on first use.
e2f_status couple_of(e2f_ctx* ctx, int L, int groups, const e2f_ctx::Couple*& out) {
  auto key = std::make_pair(L, groups);
  auto it = ctx->couple.find(key);
  if (it == ctx->couple.end()) {
    const CoupleSchedule cs = couple_schedule(ctx->host[L], groups);
    e2f_ctx::Couple c;
    c.k = cs.k;
    E2F_HIP(hipMalloc((void**)&c.meta, sizeof(int) * std::max<size_t>(cs.meta.size(), 1)));
    E2F_HIP(hipMalloc((void**)&c.coef, sizeof(float) * std::max<size_t>(cs.coef.size(), 1)));
    E2F_HIP(hipMemcpy(c.meta, cs.meta.data(), sizeof(int) * cs.meta.size(), hipMemcpyHostToDevice));
    E2F_HIP(hipMemcpy(c.coef, cs.coef.data(), sizeof(float) * cs.coef.size(), hipMemcpyHostToDevice));
    if (!cs.tab.empty()) {
      c.ntab = (int)cs.tab.size();
      E2F_HIP(hipMalloc((void**)&c.pmeta, sizeof(int) * std::max<size_t>(cs.pmeta.size(), 1)));
      E2F_HIP(hipMalloc((void**)&c.tab, sizeof(float) * cs.tab.size()));
      E2F_HIP(hipMemcpy(c.pmeta, cs.pmeta.data(), sizeof(int) * cs.pmeta.size(), hipMemcpyHostToDevice));
      E2F_HIP(hipMemcpy(c.tab, cs.tab.data(), sizeof(float) * cs.tab.size(), hipMemcpyHostToDevice));
    }
    it = ctx->couple.emplace(key, c).first;
  }
  out = &it->second;
  return E2F_OK;
}

// The backward's filter-contraction schedule for (L, head width dh), uploaded
// on first use: the most filter rows per pass whose LDS (gy slice, schedule
// up to L = 4, Z) fits 40 KB, so that four workgroups share a CU; else one
// row per pass.
e2f_status geom_of(e2f_ctx* ctx, int L, int dh, const e2f_ctx::Geom*& out) {
  auto key = std::make_pair(L, dh);
  auto it = ctx->geom.find(key);
  if (it == ctx->geom.end()) {
    const LayerTables& t = ctx->host[L];
    GeomSchedule gs;
    for (int qc = t.nk; qc >= 1; --qc) {
      gs = geom_schedule(t, qc);
      if (edge_geom_lds(L, dh, qc, (int)gs.meta.size()) <= 40960) break;
    }
    std::vector<int> oc;
    for (int c = 0; c < gs.nchunk; ++c) oc.push_back(gs.off[c]), oc.push_back(gs.ck[c]);
    e2f_ctx::Geom g;
    g.qc = gs.qc;
    g.tot = (int)gs.meta.size();
    E2F_HIP(hipMalloc((void**)&g.meta, sizeof(int) * std::max<size_t>(gs.meta.size(), 1)));
    E2F_HIP(hipMalloc((void**)&g.unit, sizeof(float) * std::max<size_t>(gs.unit.size(), 1)));
    E2F_HIP(hipMalloc((void**)&g.oc, sizeof(int) * std::max<size_t>(oc.size(), 1)));
    E2F_HIP(hipMemcpy(g.meta, gs.meta.data(), sizeof(int) * gs.meta.size(), hipMemcpyHostToDevice));
    E2F_HIP(hipMemcpy(g.unit, gs.unit.data(), sizeof(float) * gs.unit.size(), hipMemcpyHostToDevice));
    E2F_HIP(hipMemcpy(g.oc, oc.data(), sizeof(int) * oc.size(), hipMemcpyHostToDevice));
    it = ctx->geom.emplace(key, g).first;
  }
  out = &it->second;
  return E2F_OK;
}

e2f_status upload_tables(e2f_ctx* ctx, int L) {
  const LayerTables& t = ctx->host[L];
  std::vector<char> blob;
  std::vector<size_t> o;
  push_array(blob, o, t.a_row_start);  // 0
  push_array(blob, o, t.sh_ptr);       // 1
  push_array(blob, o, t.sh_pow);       // 2
  push_array(blob, o, t.sh_coef);      // 3
  push_array(blob, o, t.m_rowoff);     // 4
  push_array(blob, o, t.m_ptr);        // 5
  push_array(blob, o, t.m_ridx);       // 6
  push_array(blob, o, t.m_coef);       // 7
  push_array(blob, o, t.q_ncol);       // 8
  push_array(blob, o, t.q_coloff);     // 9
  push_array(blob, o, t.q_cols);       // 10
  push_array(blob, o, t.q_slotoff);    // 11
  push_array(blob, o, t.q_ptr);        // 12
  push_array(blob, o, t.q_ridx);       // 13
  push_array(blob, o, t.k_ptr);        // 14
  push_array(blob, o, t.k_ridx);       // 15
  std::vector<double> tpc(t.tp_sched.unit);
  push_array(blob, o, t.tp_sched.k);     // 16
  push_array(blob, o, t.tp_sched.off);   // 17
  push_array(blob, o, t.tp_sched.meta);  // 18
  push_array(blob, o, tpc);              // 19
  push_array(blob, o, t.rc_sched.k);     // 20
  push_array(blob, o, t.rc_sched.off);   // 21
  push_array(blob, o, t.rc_sched.meta);  // 22
  for (int f = 0; f <= L; ++f) {          // 23 + 3f .. 25 + 3f
    push_array(blob, o, t.rcf_sched[f].k);
    push_array(blob, o, t.rcf_sched[f].off);
    push_array(blob, o, t.rcf_sched[f].meta);
  }
  const size_t oag = o.size();
  push_array(blob, o, t.ag_ptr);          // oag
  push_array(blob, o, t.ag_idx);          // oag + 1
  push_array(blob, o, t.ag_coef);         // oag + 2
  push_array(blob, o, t.sh_dense);        // oag + 3
  void* mem = nullptr;
  E2F_HIP(hipMalloc(&mem, blob.size()));
  ctx->table_mem[L] = mem;
  E2F_HIP(hipMemcpy(mem, blob.data(), blob.size(), hipMemcpyHostToDevice));
  char* b = (char*)mem;
  DevTables d{};
  d.L = L;
  d.nk = t.nk;
  d.dimT = t.dimT;
  d.a_row_start = (const int*)(b + o[0]);
  d.sh_ptr = (const int*)(b + o[1]);
  d.sh_pow = (const int*)(b + o[2]);
  d.sh_coef = (const double*)(b + o[3]);
  d.m_rowoff = (const int*)(b + o[4]);
  d.m_ptr = (const int*)(b + o[5]);
  d.m_ridx = (const int*)(b + o[6]);
  d.m_coef = (const double*)(b + o[7]);
  d.q_ncol = (const int*)(b + o[8]);
  d.q_coloff = (const int*)(b + o[9]);
  d.q_cols = (const int*)(b + o[10]);
  d.q_slotoff = (const int*)(b + o[11]);
  d.q_ptr = (const int*)(b + o[12]);
  d.q_ridx = (const int*)(b + o[13]);
  d.k_ptr = (const int*)(b + o[14]);
  d.k_ridx = (const int*)(b + o[15]);
  d.tp_k = (const int*)(b + o[16]);
  d.tp_off = (const int*)(b + o[17]);
  d.tp_meta = (const int*)(b + o[18]);
  d.tp_coef = (const double*)(b + o[19]);
  d.rc_k = (const int*)(b + o[20]);
  d.rc_off = (const int*)(b + o[21]);
  d.rc_meta = (const int*)(b + o[22]);
  d.rc_coef = nullptr;
  d.ag_ptr = (const int*)(b + o[oag]);
  d.ag_idx = (const int*)(b + o[oag + 1]);
  d.ag_coef = (const float*)(b + o[oag + 2]);
  d.sh_dense = (const double*)(b + o[oag + 3]);
  ctx->rcf_k[L].assign(L + 1, nullptr);
  ctx->rcf_off[L].assign(L + 1, nullptr);
  ctx->rcf_meta[L].assign(L + 1, nullptr);
  for (int f = 0; f <= L; ++f) {
    ctx->rcf_k[L][f] = (const int*)(b + o[23 + 3 * f]);
    ctx->rcf_off[L][f] = (const int*)(b + o[24 + 3 * f]);
    ctx->rcf_meta[L][f] = (const int*)(b + o[25 + 3 * f]);
  }
  d.q_coef = nullptr;
  d.k_coef = nullptr;
  d.w_f = nullptr;
  d.max_qslots = t.max_qslots;
  d.m_slots = t.m_slots();
  for (int a = 0; a <= L; ++a) d.tp_rs[a] = t.tp_rs[a];
  for (int a = 0; a <= L + 1; ++a) d.tp_mo[a] = t.tp_mo[a];
  ctx->dev[L] = d;
  return E2F_OK;
}

std::vector<double> path_weights(const e2f_conv_params* p) {
  const int L1 = p->lmax + 1;
  std::vector<double> w((size_t)L1 * L1 * L1, 0.0);
  if (p->path_w) {
    std::memcpy(w.data(), p->path_w, sizeof(double) * w.size());
  } else {
    for (int a = 0; a < L1; ++a)
      for (int f = 0; f < L1; ++f)
        for (int o = std::abs(a - f); o <= std::min(a + f, p->lmax); ++o)
          w[((size_t)a * L1 + f) * L1 + o] = std::pow((double)p->cutoff, -(double)f);
  }
  return w;
}

constexpr size_t kMaxCoefSets = 16;

// The coefficient set of degree L for the path weights w: found among the
// resident sets, else built and uploaded (a synchronous upload, on first use
// only; allow_upload = false makes a missing set an error instead).
e2f_status coef_of(e2f_ctx* ctx, int L, const std::vector<double>& w, bool allow_upload,
                   const e2f_ctx::CoefSet*& out) {
  std::vector<e2f_ctx::CoefSet>& sets = ctx->coefs[L];
  for (const e2f_ctx::CoefSet& c : sets)
    if (c.w == w) {
      out = &c;
      return E2F_OK;
    }
  if (!allow_upload)
    return fail(E2F_EINVAL, "these path weights are not resident on the context; call e2f_wigner6j_prepare first");
  const LayerTables& t = ctx->host[L];
  std::vector<double> q(t.q_unit.size());
  for (size_t e = 0; e < q.size(); ++e) q[e] = t.q_unit[e] * w[t.q_path[e]];
  std::vector<float> k(t.k_unit.size());
  for (size_t e = 0; e < k.size(); ++e) k[e] = (float)(t.k_unit[e] * w[t.k_path[e]]);
  std::vector<double> rc(t.rc_sched.unit.size());
  for (size_t e = 0; e < rc.size(); ++e) rc[e] = t.rc_sched.path[e] < 0 ? 0.0 : t.rc_sched.unit[e] * w[t.rc_sched.path[e]];
  std::vector<char> blob;
  std::vector<size_t> o;
  push_array(blob, o, q);
  push_array(blob, o, k);
  push_array(blob, o, rc);
  for (int f = 0; f <= L; ++f) {  // o[3 + f]
    const Schedule& sf = t.rcf_sched[f];
    std::vector<double> c(sf.unit.size());
    for (size_t e = 0; e < c.size(); ++e) c[e] = sf.path[e] < 0 ? 0.0 : sf.unit[e] * w[sf.path[e]];
    push_array(blob, o, c);
  }
  std::vector<float> wf(w.begin(), w.end());  // o[4 + L]
  push_array(blob, o, wf);
  const int all_degs[1] = {-1};
  const FuseTable ft = fuse_table(t, w, all_degs, 1, t.nk);  // o[5 + L] .. o[7 + L] (empty above kFuseMaxL)
  push_array(blob, o, ft.ptr);
  push_array(blob, o, ft.idx);
  push_array(blob, o, ft.coef);
  YnormPass yps[kYnormMaxPasses];  // o[8 + L + 3q] .. o[10 + L + 3q]
  const int nyp = ft.coef.empty() ? 0 : ynorm_passes(L, yps);
  for (int q = 0; q < nyp; ++q) {
    const FuseTable fp = fuse_table(t, w, yps[q].degs, yps[q].nd, fuse_krows(t.nk, yps[q].degs, yps[q].nd));
    push_array(blob, o, fp.ptr);
    push_array(blob, o, fp.idx);
    push_array(blob, o, fp.coef);
  }
  if (sets.size() >= kMaxCoefSets) {  // the oldest set may still be read by queued work
    E2F_HIP(hipDeviceSynchronize());
    E2F_HIP(hipFree(sets.front().mem));
    sets.erase(sets.begin());
  }
  void* mem = nullptr;
  E2F_HIP(hipMalloc(&mem, blob.size()));
  if (hipMemcpy(mem, blob.data(), blob.size(), hipMemcpyHostToDevice) != hipSuccess) {
    (void)hipFree(mem);
    return fail(E2F_EDEVICE, "coefficient upload failed");
  }
  e2f_ctx::CoefSet c;
  c.w = w;
  c.mem = mem;
  c.q_coef = (const double*)((char*)mem + o[0]);
  c.k_coef = (const float*)((char*)mem + o[1]);
  c.rc_coef = (const double*)((char*)mem + o[2]);
  for (int f = 0; f <= L; ++f) c.rcf_coef.push_back((const double*)((char*)mem + o[3 + f]));
  c.w_f = (const float*)((char*)mem + o[4 + L]);
  if (!ft.coef.empty()) {
    auto tab = [&](size_t k, int nkr) {
      return e2f_ctx::CoefSet::FuseTab{(const int*)((char*)mem + o[k]), (const int*)((char*)mem + o[k + 1]),
                                       (const double*)((char*)mem + o[k + 2]), nkr};
    };
    c.f = tab(5 + L, t.nk);
    for (int q = 0; q < nyp; ++q) c.fy.push_back(tab(8 + L + 3 * q, fuse_krows(t.nk, yps[q].degs, yps[q].nd)));
  }
  sets.push_back(std::move(c));
  out = &sets.back();
  return E2F_OK;
}

// The device tables of degree L with the coefficients of one weight set.
DevTables with_coef(const e2f_ctx* ctx, int L, const e2f_ctx::CoefSet& c) {
  DevTables t = ctx->dev[L];
  t.q_coef = c.q_coef;
  t.k_coef = c.k_coef;
  t.rc_coef = c.rc_coef;
  t.w_f = c.w_f;
  return t;
}

// The same restricted to the recouple terms of filter degree f.
DevTables with_coef_f(const e2f_ctx* ctx, int L, const e2f_ctx::CoefSet& c, int f) {
  DevTables t = with_coef(ctx, L, c);
  t.rc_k = ctx->rcf_k[L][f];
  t.rc_off = ctx->rcf_off[L][f];
  t.rc_meta = ctx->rcf_meta[L][f];
  t.rc_coef = c.rcf_coef[f];
  return t;
}

bool finite_pos(float x) { return std::isfinite(x) && x > 0.0f; }

e2f_status check_params(e2f_ctx* ctx, const e2f_conv_params* p) {
  if (!ctx) return fail(E2F_EINVAL, "ctx is NULL");
  if (!p) return fail(E2F_EINVAL, "params is NULL");
  if (p->lmax < 0 || p->lmax > kMaxL) return fail(E2F_EUNSUPPORTED, "lmax %d outside 0..%d", p->lmax, kMaxL);
  if (p->lmax > ctx->lmax_max) return fail(E2F_EINVAL, "lmax %d above the context's %d", p->lmax, ctx->lmax_max);
  if (p->channels < 1 || p->heads < 1) return fail(E2F_EINVAL, "channels and heads must be positive");
  if (p->channels % p->heads) return fail(E2F_EINVAL, "channels %d not divisible by heads %d", p->channels, p->heads);
  if (p->channels % 4 || (p->channels / p->heads) % 4 || p->channels > 1024)
    return fail(E2F_EUNSUPPORTED, "channels %d / head width %d must be multiples of 4 (channels <= 1024)",
                p->channels, p->channels / p->heads);
  if (!finite_pos(p->cutoff) || p->cutoff > 64.0f) return fail(E2F_EINVAL, "cutoff must be finite, in (0, 64]");
  if (!std::isfinite(p->tile_side) || p->tile_side < 0.0f) return fail(E2F_EINVAL, "tile_side must be finite and >= 0");
  if (p->y_norm != 0 && p->y_norm != 1) return fail(E2F_EINVAL, "y_norm must be 0 or 1");
  if (p->form < E2F_FORM_AUTO || p->form > E2F_FORM_FUSED) return fail(E2F_EINVAL, "form must be 0, 1 or 2");
  int md = 0;  // read as an int: a C caller may store any value in the enum field
  std::memcpy(&md, &p->mix_dtype, sizeof(md));
  if (md != E2F_F32 && md != E2F_BF16) return fail(E2F_EINVAL, "unknown mix_dtype");
  if (p->path_w) {
    const int L1 = p->lmax + 1;
    for (int q = 0; q < L1 * L1 * L1; ++q)
      if (!std::isfinite(p->path_w[q])) return fail(E2F_EINVAL, "path_w[%d] is not finite", q);
  }
  return E2F_OK;
}

e2f_status check_conv(e2f_ctx* ctx, const e2f_conv_params* p, const float* pos, const float* feat, int32_t n,
                      const int64_t* row_ptr, const int32_t* col_idx, int64_t n_edges, float* out) {
  if (e2f_status rs = check_params(ctx, p); rs != E2F_OK) return rs;
  if (n < 0) return fail(E2F_EINVAL, "n < 0");
  if (n_edges < 0) return fail(E2F_EINVAL, "n_edges < 0");
  if (n_edges > std::numeric_limits<int32_t>::max()) return fail(E2F_EUNSUPPORTED, "more than 2^31-1 edges");
  if (n > 0 && (!pos || !feat || !out || !row_ptr)) return fail(E2F_EINVAL, "pos, feat, out and row_ptr are required");
  if (n_edges > 0 && !col_idx) return fail(E2F_EINVAL, "col_idx is NULL with n_edges > 0");
  const double elems = (double)n * nk_of(p->lmax) * p->channels;
  if (elems > 4.0e18) return fail(E2F_EINVAL, "feature index space overflows int64");
  if (ctx->device < 0) return fail(E2F_EDEVICE, "context has no device");
  return E2F_OK;
}

// Tile plan: bounding box on the device, then the tile grid on the host.
struct TilePlan {
  int lo[3];
  int dim[3];
  int64_t span[3];
  int ncell = 1;
  int64_t n_graphs = 1;
};

e2f_status run_bbox(e2f_ctx* ctx, const float* pos, const int32_t* graph_id, int n, hipStream_t s, int st[kStatsInts]) {
  E2F_TIMED("bbox", launch_bbox(pos, graph_id, n, ctx->stats, s));
  E2F_HIP(hipMemcpyAsync(ctx->pinned, ctx->stats, sizeof(int) * kStatsInts, hipMemcpyDeviceToHost, s));
  E2F_HIP(hipStreamSynchronize(s));
  std::memcpy(st, ctx->pinned, sizeof(int) * kStatsInts);
  if (st[7] & 1) return fail(E2F_EINVAL, "a position is not finite or has |x| >= 16384 A");
  if (st[7] & 2) return fail(E2F_EINVAL, "a graph id is negative");
  return E2F_OK;
}

// Real CG tensors of (a, f, o) and (o, f, a) are proportional with the first
// and last index swapped: C[a,f,o][al][mf][m] = kappa C[o,f,a][m][mf][al].
// kappa is read off the library's own tables and the proportionality checked.
e2f_status transpose_factors(e2f_ctx* ctx, int L, const std::vector<double>*& out) {
  if ((int)ctx->kappa.size() <= L) ctx->kappa.resize(L + 1);
  std::vector<double>& k = ctx->kappa[L];
  const int L1 = L + 1;
  if (k.empty()) {
    std::vector<double> v((size_t)L1 * L1 * L1, 0.0);
    for (int a = 0; a <= L; ++a)
      for (int f = 0; f <= L; ++f)
        for (int o = std::abs(a - f); o <= std::min(a + f, L); ++o) {
          const std::vector<double> A = real_cg(a, f, o), B = real_cg(o, f, a);
          const int na = 2 * a + 1, nf = 2 * f + 1, no = 2 * o + 1;
          double num = 0.0, den = 0.0;
          for (int x = 0; x < na; ++x)
            for (int y = 0; y < nf; ++y)
              for (int z = 0; z < no; ++z) {
                const double bt = B[((size_t)z * nf + y) * na + x];
                num += A[((size_t)x * nf + y) * no + z] * bt;
                den += bt * bt;
              }
          const double kap = num / den;
          for (int x = 0; x < na; ++x)
            for (int y = 0; y < nf; ++y)
              for (int z = 0; z < no; ++z)
                if (std::fabs(A[((size_t)x * nf + y) * no + z] - kap * B[((size_t)z * nf + y) * na + x]) > 1e-12)
                  return fail(E2F_EUNSUPPORTED, "real CG (%d,%d,%d) is not a multiple of its transpose", a, f, o);
          v[((size_t)a * L1 + f) * L1 + o] = kap;
        }
    k.swap(v);
  }
  out = &k;
  return E2F_OK;
}


// ---------------------------------------------------------------- forward
// Smallest slice of receivers a workspace must hold S for.
constexpr int64_t kMinSlice = 256;

// Byte layout of the forward's workspace: the plan and per-edge arrays (a
// fixed part), then S for a slice of receivers.
struct FwdLayout {
  size_t stats = 0, dmin = 0, grid = 0, tile_of = 0, keys = 0, keys_out = 0, vals = 0, order = 0, sort_tmp = 0;
  size_t sort_b = 0, Re = 0, Rr = 0, alpha_hm = 0, erows = 0, y = 0, featq = 0, S = 0;
  size_t fixed = 0;  // bytes before S
  size_t s_row = 0;  // S bytes per receiver
  size_t total(int64_t slice) const { return fixed + s_row * (size_t)std::max<int64_t>(slice, 0); }
};

// The split of each head into channel groups of 16 with which the
// aggregation applies the recouple itself (L <= 4, head width a multiple of
// 16; with y_norm the filter degrees stacked in the K rows of one or two
// passes); 0 where the forward writes S.  The automatic choice takes the
// fused form with y_norm (the two-kernel form then aggregates once per
// degree: 20,000 atoms, L = 1 .. 4, 1.47 ms fused vs 2.16, 2.04 vs 4.74,
// 4.79 vs 9.77, 10.6 vs 34.5),
// and otherwise at L = 4 once S would outgrow the 256 MiB on-die cache
// (measured: 1,000 atoms with 32 neighbours at L = 4, S 232 MB, 0.31 ms
// split vs 0.34 fused; 2,000 atoms with 72, S 465 MB, 0.90 vs 0.84; 20,000
// with 80, 7.17 vs 6.27; at L = 3 the split form was as fast or faster at
// every size).
int fused_split(const e2f_conv_params* p, int64_t n) {
  const int dh = p->channels / p->heads;
  if (p->form == E2F_FORM_SPLIT || dh % 16 != 0) return 0;
  if (!outer_fused_supported(p->lmax, p->channels, p->channels / 16, n)) return 0;
  if (p->form == E2F_FORM_FUSED || p->y_norm) return dh / 16;
  const double s_bytes = 4.0 * (double)n * (double)node_tp_dim(p->lmax) * p->channels;
  return p->lmax == kFuseMaxL && s_bytes > 256.0 * 1024 * 1024 ? dh / 16 : 0;
}

// Floats of one receiver's F in the fused form: the largest layout among
// the forward's passes (the alpha / D^f passes stack degrees in more K
// rows).
int fused_row_floats(const e2f_conv_params* p) {
  const int L = p->lmax, nk = nk_of(L);
  int fl = fuse_stride(nk, nk);
  YnormPass yps[kYnormMaxPasses];
  const int nyp = p->y_norm && L <= kFuseMaxL ? ynorm_passes(L, yps) : 0;
  for (int q = 0; q < nyp; ++q) fl = std::max(fl, fuse_stride(nk, fuse_krows(nk, yps[q].degs, yps[q].nd)));
  return fl;
}

FwdLayout fwd_layout(const e2f_conv_params* p, int n, int64_t E, bool have_alpha) {
  const int L = p->lmax, nk = nk_of(L), C = p->channels, H = p->heads;
  const bool ynorm = p->y_norm != 0;
  FwdLayout f;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += al256(bytes);
    return at;
  };
  f.stats = take(sizeof(int) * 16);
  f.dmin = take(sizeof(unsigned));
  f.grid = take(sizeof(TileGridDev));
  f.tile_of = take(sizeof(int32_t) * (size_t)n);
  f.keys = take(sizeof(uint64_t) * (size_t)n);
  f.keys_out = take(sizeof(uint64_t) * (size_t)n);
  f.vals = take(sizeof(int32_t) * (size_t)n);
  f.order = take(sizeof(int32_t) * (size_t)n);
  f.sort_b = plan_sort_tmp_bytes(std::max(n, 1));
  f.sort_tmp = take(f.sort_b);
  f.Re = take(sizeof(float) * (size_t)(E + kEdgePad) * nk);
  f.Rr = take(sizeof(double) * (size_t)n * nk);
  const size_t na = ynorm ? (size_t)(L + 1) : (have_alpha ? 1 : 0);
  f.alpha_hm = take(sizeof(float) * ((size_t)E * H * na + kEdgePad));
  f.erows = take(sizeof(int32_t) * (size_t)E);
  f.y = take(p->mix_w ? sizeof(float) * (size_t)n * nk * C : 0);
  // the fused aggregation's copy of the features (groups of four components,
  // each value split into three bfloat16 parts: 6 bytes)
  f.featq = take(fused_split(p, n) > 0 ? sizeof(float) * (size_t)n * C * 6 * fuse_groups(L) : 0);
  f.S = off;
  f.fixed = off;
  // per receiver of a slice: F_i (fused; the largest layout of its passes) or S_i
  f.s_row = fused_split(p, n) > 0 ? sizeof(float) * (size_t)fused_row_floats(p)
                                  : al256(sizeof(float) * (size_t)node_tp_dim(L) * C);
  return f;
}

// The split of each head into hdiv channel groups (hdiv | C/H, width a
// multiple of 4) with which the aggregation's per-receiver tile fits; 0 if none.
int head_split(int L, int C, int H) {
  const int dh = C / H;
  for (int hd = 1; hd <= dh / 4; ++hd)
    if (dh % hd == 0 && (dh / hd) % 4 == 0 && outer_agg_supported(L, C, H * hd)) return hd;
  return 0;
}

// Tile side of the local origins (precision of the binomial expansion, which
// loses about eps (|p| / cutoff)^L in fp32): cutoff * (8, 8, 8, 6, 4, 3, 2).
constexpr double kTileCutoffs[kMaxL + 1] = {8.0, 8.0, 8.0, 6.0, 4.0, 3.0, 2.0};
// With alpha / D^f the edge weights no longer damp that loss: tiles then have
// a side of at most this many shortest-edge lengths, so that the largest
// ratio (|p_i| + |p_j|) / |r_ij| stays below about 1 + 2.31 sqrt(3) = 5.
constexpr double kYnormTileScale = 2.31;

e2f_status forward_impl(e2f_ctx* ctx, const e2f_conv_params* p, const float* pos, const int32_t* graph_id,
                        const float* feat, int32_t n, const int64_t* row_ptr, const int32_t* col_idx, int64_t n_edges,
                        const float* alpha, float* out, void* workspace, size_t workspace_bytes, void* stream,
                        bool allow_upload) {
  e2f_status rs = check_conv(ctx, p, pos, feat, n, row_ptr, col_idx, n_edges, out);
  if (rs != E2F_OK) return rs;
  hipStream_t s = (hipStream_t)stream;
  DeviceGuard g(ctx->device);
  const int L = p->lmax, C = p->channels, H = p->heads, nk = nk_of(L);
  const e2f_ctx::CoefSet* cs = nullptr;
  if ((rs = coef_of(ctx, L, path_weights(p), allow_upload, cs)) != E2F_OK) return rs;
  const int fsplit = fused_split(p, n);
  const int hdiv = fsplit > 0 ? fsplit : head_split(L, C, H);
  if (hdiv < 1) return fail(E2F_EUNSUPPORTED, "no head split of width %d fits the aggregation", C / H);
  const int Hv = H * hdiv, dv = C / Hv;
  const int cgroups = outer_agg_groups(L, C, Hv);
  const e2f_ctx::Couple* cpl = nullptr;
  if (fsplit == 0) {
    if (!allow_upload && ctx->couple.find(std::make_pair(L, cgroups)) == ctx->couple.end())
      return fail(E2F_EINVAL, "the coupling schedule is not resident on the context; call e2f_wigner6j_prepare first");
    if ((rs = couple_of(ctx, L, cgroups, cpl)) != E2F_OK) return rs;
  } else if (!cs->f.ptr || (p->y_norm && cs->fy.empty())) {
    return fail(E2F_EDEVICE, "the fused recouple table of L = %d is missing", L);
  }
  if (n == 0) return E2F_OK;
  const bool ynorm = p->y_norm != 0;
  const FwdLayout f = fwd_layout(p, n, n_edges, alpha != nullptr);
  if (n_edges > 0) {
    if (!workspace) return fail(E2F_EINVAL, "workspace is NULL");
    if ((uintptr_t)workspace % 256) return fail(E2F_EINVAL, "workspace must be 256-byte aligned");
    const size_t need = f.total(std::min<int64_t>(n, kMinSlice));
    if (workspace_bytes < need)
      return fail(E2F_ECAPACITY, "workspace of %zu bytes is below the minimum %zu", workspace_bytes, need);
  }
  const DevTables t = with_coef(ctx, L, *cs);
  if (n_edges == 0) {  // every receiver is isolated (a fill kernel, no memset: capture-safe)
    E2F_HIP(launch_fill(out, (int64_t)n * nk * C, 0.0f, s));
    ctx->last_slices = 0;
    return E2F_OK;
  }
  char* ws = (char*)workspace;
  int* stats = (int*)(ws + f.stats);
  unsigned* dmin = (unsigned*)(ws + f.dmin);
  TileGridDev* grid = (TileGridDev*)(ws + f.grid);
  int32_t* tile_of = (int32_t*)(ws + f.tile_of);
  int32_t* order = (int32_t*)(ws + f.order);
  float* Re = (float*)(ws + f.Re);
  double* Rr = (double*)(ws + f.Rr);
  float* alpha_hm = (alpha || ynorm) ? (float*)(ws + f.alpha_hm) : nullptr;
  float* y = p->mix_w ? (float*)(ws + f.y) : out;
  float* S = (float*)(ws + f.S);
  // ---- plan: bounding box, attention weights head-major (per filter degree
  // under alpha / D^f, with the shortest edge), tile grid, receiver order,
  // solid harmonics of the edges and receivers
  int32_t* erows = (int32_t*)(ws + f.erows);
  // (a graph of at most kPlanSmallMax atoms takes the whole plan in one
  // workgroup: box, grid, tiles and the sorted order in one launch)
  const bool small_plan = n <= kPlanSmallMax;
  // the fused form's copy of the features needs only the features: it is
  // made on the context's second stream while the plan runs on this one
  // (the fork waits for the work already queued here; the join comes before
  // the aggregation)
  float* featq = (float*)(ws + f.featq);
  if (fsplit > 0) {
    E2F_HIP(hipEventRecord(ctx->fork, s));
    E2F_HIP(hipStreamWaitEvent(ctx->side, ctx->fork, 0));
    {
      hipStream_t s = ctx->side;  // (E2F_TIMED records on s)
      E2F_TIMED("feat_qmajor", launch_feat_qmajor(L, feat, n, C, featq, s));
    }
    E2F_HIP(hipEventRecord(ctx->join, ctx->side));
  }
  if (!small_plan) E2F_TIMED("bbox", launch_plan_bbox(pos, graph_id, n, stats, ynorm ? dmin : nullptr, s));
  else if (ynorm) E2F_TIMED("bbox", launch_plan_init(stats, dmin, s));
  // (the receiver of every edge, and in the same launch the weights
  // head-major unless y_norm scales them per filter degree)
  E2F_TIMED("tile_plan", launch_plan_edge_rows(row_ptr, n, n_edges, erows, ynorm ? nullptr : alpha, H,
                                               ynorm ? nullptr : alpha_hm, s));
  if (ynorm) {
    E2F_TIMED("alpha_hm", launch_plan_dmin(pos, erows, col_idx, n, n_edges, dmin, s));
    E2F_TIMED("alpha_hm", launch_alpha_dnorm(pos, nullptr, col_idx, alpha, n, n_edges, H, L, erows, alpha_hm, s));
  }
  const double side = (p->tile_side > 0.0f ? (double)p->tile_side : kTileCutoffs[L] * (double)p->cutoff) * kGrid;
  if (small_plan) {
    E2F_TIMED("tile_plan", launch_plan_small(pos, graph_id, n, ynorm ? dmin : nullptr, side, kYnormTileScale, stats,
                                             grid, tile_of, order, s));
  } else {
    E2F_TIMED("tile_plan", launch_plan_grid(stats, ynorm ? dmin : nullptr, side, kYnormTileScale, grid, s));
    E2F_TIMED("tile_plan", launch_plan_order(pos, graph_id, n, grid, tile_of, (uint64_t*)(ws + f.keys),
                                             (uint64_t*)(ws + f.keys_out), (int32_t*)(ws + f.vals), order,
                                             ws + f.sort_tmp, f.sort_b, s));
  }
  E2F_TIMED("sh", launch_plan_sh(t, pos, erows, col_idx, n, n_edges, tile_of, grid, Rr, Re, s));
  // ---- aggregation and recouple per slice of receivers (S of one slice
  // at a time in the workspace)
  const int64_t slice = std::min<int64_t>(n, (int64_t)((workspace_bytes - f.fixed) / f.s_row));
  int64_t slices = 0;
  if (fsplit > 0) E2F_HIP(hipStreamWaitEvent(s, ctx->join, 0));
  for (int64_t q0 = 0; q0 < n; q0 += slice, ++slices) {
    const int nb = (int)std::min<int64_t>(slice, n - q0);
    const int32_t* ord = order + q0;
    if (fsplit > 0) {
      // per pass: F of the slice (from a table whose K rows stack the pass's
      // filter degrees), then the aggregation with the recouple applied; the
      // passes after the first add to y.  The plain layer: one pass.  With
      // y_norm the weights alpha / D^f and the terms b + u = f of each degree
      // f, in (f+1)^2 K rows: the passes of ynorm_passes (one below L = 4;
      // at L = 4 degrees 3 and 2, then 4, 1 and 0).
      int npass = 0;
      const int all_degs[1] = {-1};
      auto pass = [&](const e2f_ctx::CoefSet::FuseTab& tab, const int* degs, int nd) -> e2f_status {
        FusedSegs sg{};
        sg.n = nd;
        for (int q = 0, r = 0; q < nd; ++q) {
          sg.alpha_hm[q] = degs[q] < 0 ? alpha_hm : alpha_hm + (size_t)degs[q] * H * n_edges;
          sg.start[q] = r;
          r += degs[q] < 0 ? nk : (degs[q] + 1) * (degs[q] + 1);
        }
        E2F_TIMED("fuse_build", launch_fuse_build(L, tab.nkr, tab.ptr, tab.idx, tab.coef, Rr, ord, nb, S, s));
        E2F_TIMED("aggregate", launch_outer_fused(L, tab.nkr, Re, row_ptr, col_idx, sg, n_edges, featq, ord, S, nb, C,
                                                  Hv, hdiv, n, npass++ > 0, y, s));
        return E2F_OK;
      };
      if (!ynorm) {
        if ((rs = pass(cs->f, all_degs, 1)) != E2F_OK) return rs;
      } else {
        YnormPass yps[kYnormMaxPasses];
        const int nyp = ynorm_passes(L, yps);
        if (nyp != (int)cs->fy.size()) return fail(E2F_EDEVICE, "the alpha / D^f tables of L = %d are missing", L);
        for (int q = 0; q < nyp; ++q)
          if ((rs = pass(cs->fy[q], yps[q].degs, yps[q].nd)) != E2F_OK) return rs;
      }
      continue;
    }
    if (!ynorm) {
      E2F_TIMED("aggregate", launch_outer_agg(t, Re, row_ptr, col_idx, alpha_hm, n_edges, feat, ord, cpl->meta,
                                              cpl->coef, cpl->pmeta, cpl->tab, cpl->ntab, cpl->k, cgroups, nb, C, Hv,
                                              hdiv, n, S, s));
      E2F_TIMED("recouple", launch_recouple(t, Rr, S, false, ord, nb, C, dv, y, s));
      continue;
    }
    // S^(f) = sum_j alpha_ij D_ij^-f [h_j (x) R(p_j)] coupled, then the
    // recouple terms of filter degree b + u = f; the f = 0 pass stores y,
    // the others add
    for (int fd = 0; fd <= L; ++fd) {
      E2F_TIMED("aggregate", launch_outer_agg(t, Re, row_ptr, col_idx, alpha_hm + (size_t)fd * H * n_edges, n_edges,
                                              feat, ord, cpl->meta, cpl->coef, cpl->pmeta, cpl->tab, cpl->ntab,
                                              cpl->k, cgroups, nb, C, Hv, hdiv, n, S, s));
      E2F_TIMED("recouple", launch_recouple(with_coef_f(ctx, L, *cs, fd), Rr, S, false, ord, nb, C, dv, y, s, fd > 0));
    }
  }
  if (p->mix_w) E2F_TIMED("mix", launch_mix(L, y, p->mix_w, p->mix_dtype == E2F_BF16, n, C, out, s));
  ctx->last_slices = slices;
  return E2F_OK;
}
}  // namespace

extern "C" {

e2f_status e2f_create(int lmax_max, int device, e2f_ctx** out) {
  if (!out) return fail(E2F_EINVAL, "out is NULL");
  *out = nullptr;
  if (lmax_max < 0 || lmax_max > kMaxL) return fail(E2F_EINVAL, "lmax_max %d outside 0..%d", lmax_max, kMaxL);
  if (device < -1) return fail(E2F_EINVAL, "device %d", device);
  e2f_ctx* ctx = new e2f_ctx();
  ctx->device = device;
  ctx->lmax_max = lmax_max;
  for (int L = 0; L <= lmax_max; ++L) ctx->host.push_back(build_layer_tables(L));
  ctx->dev.assign(lmax_max + 1, DevTables{});
  ctx->table_mem.assign(lmax_max + 1, nullptr);
  ctx->coefs.assign(lmax_max + 1, {});
  ctx->rcf_k.assign(lmax_max + 1, {});
  ctx->rcf_off.assign(lmax_max + 1, {});
  ctx->rcf_meta.assign(lmax_max + 1, {});
  if (device >= 0) {
    int count = 0;
    if (hipGetDeviceCount(&count) != hipSuccess || device >= count) {
      (void)hipGetLastError();
      delete ctx;
      return fail(E2F_EDEVICE, "HIP device %d not available", device);
    }
    DeviceGuard g(device);
    if (!g.ok) {
      delete ctx;
      return fail(E2F_EDEVICE, "hipSetDevice(%d) failed", device);
    }
    e2f_status st = E2F_OK;
    for (int L = 0; L <= lmax_max && st == E2F_OK; ++L) st = upload_tables(ctx, L);
    if (st == E2F_OK && hipMalloc((void**)&ctx->stats, sizeof(int) * 64) != hipSuccess)
      st = fail(E2F_ENOMEM, "stats allocation failed");
    if (st == E2F_OK && hipHostMalloc((void**)&ctx->pinned, sizeof(int64_t) * 16, hipHostMallocDefault) != hipSuccess)
      st = fail(E2F_ENOMEM, "pinned allocation failed");
    if (st == E2F_OK) {  // this device's copy of the scratch array (the device is current here)
      const hipError_t e = hipGetSymbolAddress(&ctx->scratch, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !ctx->scratch) {
        ctx->scratch = nullptr;
        st = fail(E2F_EDEVICE, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
      }
    }
    if (st == E2F_OK && (hipStreamCreateWithFlags(&ctx->side, hipStreamNonBlocking) != hipSuccess ||
                         hipEventCreateWithFlags(&ctx->fork, hipEventDisableTiming) != hipSuccess ||
                         hipEventCreateWithFlags(&ctx->join, hipEventDisableTiming) != hipSuccess))
      st = fail(E2F_EDEVICE, "side stream or its events: %s", hipGetErrorString(hipGetLastError()));
    if (st != E2F_OK) {
      e2f_destroy(ctx);
      return st;
    }
  }
  *out = ctx;
  return E2F_OK;
}

void e2f_destroy(e2f_ctx* ctx) {
  if (!ctx) return;
  if (ctx->device >= 0) {
    DeviceGuard g(ctx->device);
    (void)hipDeviceSynchronize();
    for (void* p : ctx->table_mem)
      if (p) (void)hipFree(p);
    for (auto& sets : ctx->coefs)
      for (auto& c : sets)
        if (c.mem) (void)hipFree(c.mem);
    for (Buf* b : {&ctx->a, &ctx->b, &ctx->c, &ctx->d})
      if (b->p) (void)hipFree(b->p);
    for (auto& kv : ctx->couple) {
      if (kv.second.meta) (void)hipFree(kv.second.meta);
      if (kv.second.coef) (void)hipFree(kv.second.coef);
      if (kv.second.pmeta) (void)hipFree(kv.second.pmeta);
      if (kv.second.tab) (void)hipFree(kv.second.tab);
    }
    for (auto& kv : ctx->geom) {
      if (kv.second.meta) (void)hipFree(kv.second.meta);
      if (kv.second.unit) (void)hipFree(kv.second.unit);
      if (kv.second.oc) (void)hipFree(kv.second.oc);
    }
    for (auto& r : ctx->recs) {
      ctx->pool.push_back(r.start);
      ctx->pool.push_back(r.stop);
    }
    for (hipEvent_t e : ctx->pool) (void)hipEventDestroy(e);
    if (ctx->fork) (void)hipEventDestroy(ctx->fork);
    if (ctx->join) (void)hipEventDestroy(ctx->join);
    if (ctx->side) (void)hipStreamDestroy(ctx->side);
    if (ctx->stats) (void)hipFree(ctx->stats);
    if (ctx->pinned) (void)hipHostFree(ctx->pinned);
    if (ctx->pinned_plan) (void)hipHostFree(ctx->pinned_plan);
  }
  delete ctx;
}

const char* e2f_last_error(void) { return g_err.c_str(); }

int64_t e2f_node_tp_dim(int lmax) { return node_tp_dim(lmax); }

e2f_status e2f_real_cg(int l1, int l2, int l3, double* out) {
  if (!out) return fail(E2F_EINVAL, "out is NULL");
  if (l1 < 0 || l2 < 0 || l3 < 0 || l1 > 12 || l2 > 12 || l3 > 12) return fail(E2F_EINVAL, "degrees must be in 0..12");
  if (l3 < std::abs(l1 - l2) || l3 > l1 + l2) return fail(E2F_EINVAL, "(%d,%d,%d) violates the triangle rule", l1, l2, l3);
  std::vector<double> c = real_cg(l1, l2, l3);
  std::memcpy(out, c.data(), sizeof(double) * c.size());
  return E2F_OK;
}

double e2f_recoupling_weight(int a, int b, int u, int o, int d) {
  if (a < 0 || b < 0 || u < 0 || o < 0 || d < 0 || a > 12 || b > 12 || u > 12 || o > 12 || d > 24) return 0.0;
  return recoupling_weight(a, b, u, o, d);
}

e2f_status e2f_neighbor_list(e2f_ctx* ctx, const float* pos, const int32_t* graph_id, int32_t n, float cutoff,
                             int64_t* row_ptr, int32_t* col_idx, int64_t capacity, int64_t* n_edges, void* stream) {
  if (!ctx) return fail(E2F_EINVAL, "ctx is NULL");
  if (!row_ptr || !n_edges) return fail(E2F_EINVAL, "row_ptr and n_edges are required");
  if (n < 0) return fail(E2F_EINVAL, "n < 0");
  if (n > 0 && !pos) return fail(E2F_EINVAL, "pos is NULL");
  if (!finite_pos(cutoff) || cutoff > 64.0f) return fail(E2F_EINVAL, "cutoff must be finite, in (0, 64]");
  if (capacity < 0) return fail(E2F_EINVAL, "capacity < 0");
  if (ctx->device < 0) return fail(E2F_EDEVICE, "context has no device");
  hipStream_t s = (hipStream_t)stream;
  DeviceGuard g(ctx->device);
  if (n == 0) {
    E2F_HIP(hipMemsetAsync(row_ptr, 0, sizeof(int64_t), s));
    E2F_HIP(hipStreamSynchronize(s));
    *n_edges = 0;
    return col_idx ? E2F_OK : fail(E2F_ECAPACITY, "size query: 0 edges");
  }
  int st[kStatsInts];
  e2f_status rs = run_bbox(ctx, pos, graph_id, n, s, st);
  if (rs != E2F_OK) return rs;
  CellGrid cg;
  const double rc = (double)cutoff * kGrid;
  cg.side = (int64_t)std::ceil(rc);
  const int64_t limit = std::max<int64_t>(8 * (int64_t)n, 4096);
  for (;;) {
    cg.ncell = 1;
    for (int k = 0; k < 3; ++k) {
      cg.lo[k] = st[k];
      cg.dim[k] = (int)(((int64_t)st[3 + k] - st[k]) / cg.side + 1);
      cg.ncell *= cg.dim[k];
    }
    if (cg.ncell <= limit) break;
    cg.side *= 2;
  }
  rs = ensure(ctx, ctx->a, nl_scratch_bytes(n, cg), s);
  if (rs != E2F_OK) return rs;
  E2F_TIMED("nl_count", launch_nl_count(pos, graph_id, n, rc * rc, cg, ctx->a.p, row_ptr, ctx->stats + 9, s));
  E2F_HIP(hipMemcpyAsync(ctx->pinned, row_ptr + n, sizeof(int64_t), hipMemcpyDeviceToHost, s));
  E2F_HIP(hipMemcpyAsync(ctx->pinned + 1, ctx->stats + 9, sizeof(int), hipMemcpyDeviceToHost, s));
  E2F_HIP(hipStreamSynchronize(s));
  const int64_t E = ctx->pinned[0];
  int max_degree = 0;
  std::memcpy(&max_degree, ctx->pinned + 1, sizeof(int));
  *n_edges = E;
  if (!col_idx || E > capacity) return fail(E2F_ECAPACITY, "the graph has %lld edges", (long long)E);
  if (E > std::numeric_limits<int32_t>::max()) return fail(E2F_EUNSUPPORTED, "more than 2^31-1 edges");
  if (E == 0) return E2F_OK;
  const size_t sort_b = nl_sort_tmp_bytes(n, E);
  rs = ensure(ctx, ctx->b, al256(sizeof(int32_t) * (size_t)E) + al256(sort_b), s);
  if (rs != E2F_OK) return rs;
  Carver cv{(char*)ctx->b.p};
  int32_t* unsorted = cv.take<int32_t>((size_t)E);
  void* sort_tmp = cv.take<char>(sort_b);
  E2F_TIMED("nl_fill", launch_nl_fill(pos, graph_id, n, rc * rc, cg, ctx->a.p, row_ptr, unsorted, col_idx, E,
                                      max_degree, sort_tmp, sort_b, s));
  return E2F_OK;
}

e2f_status e2f_knn_graph(e2f_ctx* ctx, const float* pos, const int32_t* graph_id, int32_t n, int32_t k,
                         int64_t* row_ptr, int32_t* col_idx, int64_t capacity, int64_t* n_edges, void* stream) {
  if (!ctx) return fail(E2F_EINVAL, "ctx is NULL");
  if (!row_ptr || !n_edges) return fail(E2F_EINVAL, "row_ptr and n_edges are required");
  if (n < 0) return fail(E2F_EINVAL, "n < 0");
  if (n > 0 && !pos) return fail(E2F_EINVAL, "pos is NULL");
  if (k < 1) return fail(E2F_EINVAL, "k = %d < 1", k);
  if (k > kKnnMaxK) return fail(E2F_EUNSUPPORTED, "k = %d > %d", k, kKnnMaxK);
  if (capacity < 0) return fail(E2F_EINVAL, "capacity < 0");
  if (ctx->device < 0) return fail(E2F_EDEVICE, "context has no device");
  hipStream_t s = (hipStream_t)stream;
  DeviceGuard g(ctx->device);
  if (n == 0) {
    E2F_HIP(hipMemsetAsync(row_ptr, 0, sizeof(int64_t), s));
    E2F_HIP(hipStreamSynchronize(s));
    *n_edges = 0;
    return col_idx ? E2F_OK : fail(E2F_ECAPACITY, "size query: 0 edges");
  }
  int st[kStatsInts];
  e2f_status rs = run_bbox(ctx, pos, graph_id, n, s, st);
  if (rs != E2F_OK) return rs;
  const int64_t ngraph = graph_id ? (int64_t)st[6] + 1 : 1;
  if (ngraph > (int64_t)1 << 24) return fail(E2F_EUNSUPPORTED, "graph ids above 2^24");
  rs = ensure(ctx, ctx->a, knn_scratch_bytes(n, (int)ngraph), s);
  if (rs != E2F_OK) return rs;
  E2F_TIMED("knn", launch_knn_count(graph_id, n, k, (int)ngraph, ctx->a.p, row_ptr, s));
  E2F_HIP(hipMemcpyAsync(ctx->pinned, row_ptr + n, sizeof(int64_t), hipMemcpyDeviceToHost, s));
  E2F_HIP(hipStreamSynchronize(s));
  const int64_t E = ctx->pinned[0];
  *n_edges = E;
  if (!col_idx || E > capacity) return fail(E2F_ECAPACITY, "the graph has %lld edges", (long long)E);
  if (E > std::numeric_limits<int32_t>::max()) return fail(E2F_EUNSUPPORTED, "more than 2^31-1 edges");
  if (E == 0) return E2F_OK;
  E2F_TIMED("knn", launch_knn_fill(pos, graph_id, n, k, row_ptr, col_idx, s));
  return E2F_OK;
}

e2f_status e2f_attention_weights(e2f_ctx* ctx, const float* pos, const float* q, const float* k, int32_t n,
                                 int32_t heads, int32_t dk, const float* rbf_w, int32_t n_rbf, float cutoff,
                                 const int64_t* row_ptr, const int32_t* col_idx, int64_t n_edges, float* alpha,
                                 void* stream) {
  if (!ctx) return fail(E2F_EINVAL, "ctx is NULL");
  if (n < 0 || n_edges < 0) return fail(E2F_EINVAL, "n or n_edges < 0");
  if (heads < 1) return fail(E2F_EINVAL, "heads = %d < 1", heads);
  if (heads > 64) return fail(E2F_EUNSUPPORTED, "heads = %d > 64", heads);
  if (dk < 0 || n_rbf < 0 || n_rbf == 1) return fail(E2F_EINVAL, "dk >= 0 and n_rbf = 0 or >= 2 are required");
  if (n_rbf > kAttnMaxRbf) return fail(E2F_EUNSUPPORTED, "n_rbf = %d > %d", n_rbf, kAttnMaxRbf);
  if (!finite_pos(cutoff)) return fail(E2F_EINVAL, "cutoff must be finite and positive");
  if (n > 0 && (!pos || !row_ptr)) return fail(E2F_EINVAL, "pos and row_ptr are required");
  if (n > 0 && dk > 0 && (!q || !k)) return fail(E2F_EINVAL, "q and k are required with dk > 0");
  if (n_rbf > 0 && !rbf_w) return fail(E2F_EINVAL, "rbf_w is required with n_rbf > 0");
  if (n_edges > 0 && (!col_idx || !alpha)) return fail(E2F_EINVAL, "col_idx and alpha are required");
  if (n_edges > std::numeric_limits<int32_t>::max()) return fail(E2F_EUNSUPPORTED, "more than 2^31-1 edges");
  if (ctx->device < 0) return fail(E2F_EDEVICE, "context has no device");
  if (n == 0 || n_edges == 0) return E2F_OK;
  hipStream_t s = (hipStream_t)stream;
  DeviceGuard g(ctx->device);
  E2F_TIMED("attention", launch_attention(pos, q, k, n, heads, dk, rbf_w, n_rbf, cutoff, row_ptr, col_idx, alpha, s));
  return E2F_OK;
}

e2f_status e2f_solid_harmonics(e2f_ctx* ctx, const float* pos, const float* origins, const int32_t* origin_id,
                               int32_t n, int lmax, float* out, void* stream) {
  if (!ctx) return fail(E2F_EINVAL, "ctx is NULL");
  if (lmax < 0 || lmax > ctx->lmax_max) return fail(E2F_EINVAL, "lmax %d outside 0..%d", lmax, ctx->lmax_max);
  if (n < 0) return fail(E2F_EINVAL, "n < 0");
  if (n > 0 && (!pos || !out)) return fail(E2F_EINVAL, "pos and out are required");
  if (ctx->device < 0) return fail(E2F_EDEVICE, "context has no device");
  if (n == 0) return E2F_OK;
  hipStream_t s = (hipStream_t)stream;
  DeviceGuard g(ctx->device);
  E2F_HIP(launch_sh(ctx->dev[lmax], pos, nullptr, nullptr, origins, origin_id, std::numeric_limits<int>::max(), n,
                    nullptr, out, s));
  return E2F_OK;
}

e2f_status e2f_node_tp(e2f_ctx* ctx, const float* pos, const float* origins, const int32_t* origin_id,
                       const float* feat, int32_t n, int32_t channels, int lmax, float* out, void* stream) {
  if (!ctx) return fail(E2F_EINVAL, "ctx is NULL");
  if (lmax < 0 || lmax > ctx->lmax_max) return fail(E2F_EINVAL, "lmax %d outside 0..%d", lmax, ctx->lmax_max);
  if (n < 0) return fail(E2F_EINVAL, "n < 0");
  if (channels < 4 || channels % 4 || channels > 1024)
    return fail(E2F_EUNSUPPORTED, "channels %d must be a multiple of 4 in 4..1024", channels);
  if (n > 0 && (!pos || !feat || !out)) return fail(E2F_EINVAL, "pos, feat and out are required");
  if (ctx->device < 0) return fail(E2F_EDEVICE, "context has no device");
  if (n == 0) return E2F_OK;
  hipStream_t s = (hipStream_t)stream;
  DeviceGuard g(ctx->device);
  const DevTables& t = ctx->dev[lmax];
  e2f_status rs = ensure(ctx, ctx->c, sizeof(double) * (size_t)n * t.nk, s);
  if (rs != E2F_OK) return rs;
  double* R = (double*)ctx->c.p;
  E2F_HIP(launch_sh(t, pos, nullptr, nullptr, origins, origin_id, std::numeric_limits<int>::max(), n, R, nullptr, s));
  E2F_HIP(launch_node_tp(t, R, nullptr, feat, n, channels, channels, out, s));
  return E2F_OK;
}

e2f_status e2f_wigner6j_workspace_size(e2f_ctx* ctx, const e2f_conv_params* p, int32_t n, int64_t n_edges,
                                       size_t* bytes) {
  if (!bytes) return fail(E2F_EINVAL, "bytes is NULL");
  if (e2f_status rs = check_params(ctx, p); rs != E2F_OK) return rs;
  if (n < 0 || n_edges < 0) return fail(E2F_EINVAL, "n or n_edges < 0");
  *bytes = fwd_layout(p, n, n_edges, true).total(n);
  return E2F_OK;
}

e2f_status e2f_wigner6j_workspace_min(e2f_ctx* ctx, const e2f_conv_params* p, int32_t n, int64_t n_edges,
                                      size_t* bytes) {
  if (!bytes) return fail(E2F_EINVAL, "bytes is NULL");
  if (e2f_status rs = check_params(ctx, p); rs != E2F_OK) return rs;
  if (n < 0 || n_edges < 0) return fail(E2F_EINVAL, "n or n_edges < 0");
  *bytes = fwd_layout(p, n, n_edges, true).total(std::min<int64_t>(n, kMinSlice));
  return E2F_OK;
}

e2f_status e2f_wigner6j_prepare(e2f_ctx* ctx, const e2f_conv_params* p) {
  if (e2f_status rs = check_params(ctx, p); rs != E2F_OK) return rs;
  if (ctx->device < 0) return fail(E2F_EDEVICE, "context has no device");
  DeviceGuard g(ctx->device);
  const e2f_ctx::CoefSet* cs = nullptr;
  if (e2f_status rs = coef_of(ctx, p->lmax, path_weights(p), true, cs); rs != E2F_OK) return rs;
  // the coupling schedule of the two-kernel form as well (the forward takes
  // it for atom counts whose re-laid features exceed 32-bit offsets); the
  // fused table is part of the coefficient set
  const int hdiv = head_split(p->lmax, p->channels, p->heads);
  if (hdiv < 1) {
    e2f_conv_params pf = *p;
    pf.form = E2F_FORM_FUSED;
    if (fused_split(&pf, 1) > 0) return E2F_OK;
    return fail(E2F_EUNSUPPORTED, "no head split of width %d fits the aggregation", p->channels / p->heads);
  }
  const e2f_ctx::Couple* cpl = nullptr;
  return couple_of(ctx, p->lmax, outer_agg_groups(p->lmax, p->channels, p->heads * hdiv), cpl);
}

e2f_status e2f_wigner6j_conv_forward(e2f_ctx* ctx, const e2f_conv_params* p, const float* pos,
                                     const int32_t* graph_id, const float* feat, int32_t n, const int64_t* row_ptr,
                                     const int32_t* col_idx, int64_t n_edges, const float* alpha, float* out,
                                     void* workspace, size_t workspace_bytes, void* stream) {
  return forward_impl(ctx, p, pos, graph_id, feat, n, row_ptr, col_idx, n_edges, alpha, out, workspace,
                      workspace_bytes, stream, true);
}

e2f_status e2f_wigner6j_conv_forward_noalloc(e2f_ctx* ctx, const e2f_conv_params* p, const float* pos,
                                             const int32_t* graph_id, const float* feat, int32_t n,
                                             const int64_t* row_ptr, const int32_t* col_idx, int64_t n_edges,
                                             const float* alpha, float* out, void* stream) {
  if (e2f_status rs = check_conv(ctx, p, pos, feat, n, row_ptr, col_idx, n_edges, out); rs != E2F_OK) return rs;
  if (!ctx->scratch) return fail(E2F_EDEVICE, "the context has no scratch memory");
  const size_t need = fwd_layout(p, n, n_edges, alpha != nullptr).total(std::min<int64_t>(n, kMinSlice));
  if (n_edges > 0 && need > kScratchBytes)
    return fail(E2F_ECAPACITY, "the forward needs at least %zu bytes of workspace; the scratch memory holds %zu",
                need, kScratchBytes);
  // no upload: the coefficient set and coupling schedule must be resident
  return forward_impl(ctx, p, pos, graph_id, feat, n, row_ptr, col_idx, n_edges, alpha, out, ctx->scratch,
                      kScratchBytes, stream, false);
}

e2f_status e2f_validate_graph(e2f_ctx* ctx, int32_t n, const int64_t* row_ptr, const int32_t* col_idx,
                              int64_t n_edges, int32_t* bad, void* stream) {
  if (!ctx || !bad) return fail(E2F_EINVAL, "ctx and bad are required");
  if (n < 0 || n_edges < 0) return fail(E2F_EINVAL, "n or n_edges < 0");
  if (!row_ptr) return fail(E2F_EINVAL, "row_ptr is required");
  if (n_edges > 0 && !col_idx) return fail(E2F_EINVAL, "col_idx is NULL with n_edges > 0");
  if (ctx->device < 0) return fail(E2F_EDEVICE, "context has no device");
  hipStream_t s = (hipStream_t)stream;
  DeviceGuard g(ctx->device);
  E2F_HIP(launch_validate_graph(row_ptr, col_idx, n, n_edges, ctx->stats + 16, s));
  E2F_HIP(hipMemcpyAsync(ctx->pinned, ctx->stats + 16, sizeof(int), hipMemcpyDeviceToHost, s));
  E2F_HIP(hipStreamSynchronize(s));
  int v = 0;
  std::memcpy(&v, ctx->pinned, sizeof(int));
  *bad = v;
  return E2F_OK;
}

// ---------------------------------------------------------------- standalone aggregation
namespace {
struct A3Layout {
  size_t order = 0, blk_count = 0, blk_off = 0, ucount = 0, uni = 0, edge_slot = 0, alpha_hm = 0, tmp = 0;
  size_t tmp_b = 0, total = 0;
};
A3Layout a3_layout(int n, int64_t E, int H) {
  const int nblk = (n + 15) / 16;
  A3Layout f;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += al256(bytes);
    return at;
  };
  f.order = take(sizeof(int32_t) * (size_t)n);
  f.blk_count = take(sizeof(int32_t) * (size_t)(nblk + 1));
  f.blk_off = take(sizeof(int32_t) * (size_t)(nblk + 1));
  f.ucount = take(sizeof(int32_t) * (size_t)(nblk + 1));
  f.uni = take(sizeof(int32_t) * (size_t)E);
  f.edge_slot = take(sizeof(int32_t) * (size_t)E);
  f.alpha_hm = take(sizeof(float) * (size_t)E * H);
  f.tmp_b = blocks_tmp_bytes(std::max(nblk, 1));
  f.tmp = take(f.tmp_b);
  f.total = off;
  return f;
}

e2f_status check_a3(int32_t n, int32_t rows, int32_t channels, int32_t heads, int64_t n_edges) {
  if (n < 0 || n_edges < 0) return fail(E2F_EINVAL, "n or n_edges < 0");
  if (rows < 1 || channels < 1 || heads < 1) return fail(E2F_EINVAL, "rows, channels and heads must be positive");
  if (channels % heads || (channels / heads) % 4)
    return fail(E2F_EINVAL, "channels %d must split into heads of a multiple of 4 channels", channels);
  if (n_edges >= ((int64_t)1 << 31)) return fail(E2F_EUNSUPPORTED, "n_edges must be below 2^31");
  if ((double)n * rows * channels > 4.0e18) return fail(E2F_EINVAL, "index space overflows int64");
  return E2F_OK;
}
}  // namespace

e2f_status e2f_aggregate_workspace_size(e2f_ctx* ctx, int32_t n, int64_t n_edges, int32_t heads, size_t* bytes) {
  if (!ctx || !bytes) return fail(E2F_EINVAL, "ctx and bytes are required");
  if (e2f_status rs = check_a3(n, 1, 4 * std::max(heads, 1), heads, n_edges); rs != E2F_OK) return rs;
  *bytes = a3_layout(n, n_edges, heads).total;
  return E2F_OK;
}

e2f_status e2f_aggregate(e2f_ctx* ctx, const float* T, int32_t n, int32_t rows, int32_t channels, int32_t heads,
                         const int64_t* row_ptr, const int32_t* col_idx, int64_t n_edges, const float* alpha,
                         const int32_t* order_in, float* S, void* workspace, size_t workspace_bytes, void* stream) {
  if (!ctx) return fail(E2F_EINVAL, "ctx is NULL");
  if (e2f_status rs = check_a3(n, rows, channels, heads, n_edges); rs != E2F_OK) return rs;
  if (!T || !S || !row_ptr) return fail(E2F_EINVAL, "T, S and row_ptr are required");
  if (n_edges > 0 && !col_idx) return fail(E2F_EINVAL, "col_idx is NULL with n_edges > 0");
  if (ctx->device < 0) return fail(E2F_EDEVICE, "context has no device");
  hipStream_t s = (hipStream_t)stream;
  DeviceGuard g(ctx->device);
  if (n == 0) return E2F_OK;
  if (n_edges == 0) {  // every receiver is isolated
    E2F_HIP(launch_fill(S, (int64_t)n * rows * channels, 0.0f, s));
    return E2F_OK;
  }
  const A3Layout f = a3_layout(n, n_edges, heads);
  if (!workspace) return fail(E2F_EINVAL, "workspace is NULL");
  if ((uintptr_t)workspace % 256) return fail(E2F_EINVAL, "workspace must be 256-byte aligned");
  if (workspace_bytes < f.total)
    return fail(E2F_ECAPACITY, "workspace of %zu bytes is below the required %zu", workspace_bytes, f.total);
  char* ws = (char*)workspace;
  int32_t* order = (int32_t*)(ws + f.order);
  int* bad = ctx->stats + 24;
  int* maxc = ctx->stats + 25;
  // the graph checks and the largest block, read back once
  E2F_TIMED("a3_plan", launch_validate_graph(row_ptr, col_idx, n, n_edges, bad, s));
  E2F_TIMED("a3_plan", launch_a3_checks(row_ptr, col_idx, n, n_edges, bad, maxc, s));
  if (order_in) E2F_TIMED("a3_plan", launch_a3_order_check(order_in, n, order, bad, s));  // order's space as scratch
  E2F_HIP(hipMemcpyAsync(ctx->pinned, bad, 2 * sizeof(int), hipMemcpyDeviceToHost, s));
  E2F_HIP(hipStreamSynchronize(s));
  int st[2];
  std::memcpy(st, ctx->pinned, sizeof(st));
  if (st[0]) return fail(E2F_EINVAL, "malformed graph (bits %d: 1 row_ptr[0], 2 decreasing row_ptr, 4 row_ptr[n], "
                         "8 sender out of range, 16 senders of a row not strictly ascending, 32 order not a "
                         "permutation)", st[0]);
  const bool blocks = st[1] <= a3_union_max();
  float* alpha_hm = alpha ? (float*)(ws + f.alpha_hm) : nullptr;
  if (order_in) E2F_HIP(hipMemcpyAsync(order, order_in, sizeof(int32_t) * (size_t)n, hipMemcpyDeviceToDevice, s));
  else E2F_TIMED("a3_plan", launch_iota(n, order, s));
  if (alpha && blocks) E2F_TIMED("a3_plan", launch_alpha_head_major(alpha, n_edges, heads, alpha_hm, s));
  int32_t* blk_count = (int32_t*)(ws + f.blk_count);
  int32_t* blk_off = (int32_t*)(ws + f.blk_off);
  int32_t* ucount = (int32_t*)(ws + f.ucount);
  int32_t* uni = (int32_t*)(ws + f.uni);
  int32_t* edge_slot = (int32_t*)(ws + f.edge_slot);
  if (blocks)
    E2F_TIMED("a3_plan", launch_block_union(row_ptr, col_idx, order, n, blk_count, blk_off, uni, ucount, edge_slot,
                                            ws + f.tmp, f.tmp_b, s));
  E2F_TIMED("a3_aggregate", launch_aggregate(T, 0, row_ptr, col_idx, alpha, alpha_hm, n_edges, n, order, uni, blk_off,
                                             ucount, edge_slot, blocks, n, rows, channels, heads, S, s));
  return E2F_OK;
}

e2f_status e2f_edge_tp_conv_forward(e2f_ctx* ctx, const e2f_conv_params* p, const float* pos,
                                    const int32_t* graph_id, const float* feat, int32_t n, const int64_t* row_ptr,
                                    const int32_t* col_idx, int64_t n_edges, const float* alpha, float* out,
                                    void* stream) {
  (void)graph_id;
  e2f_status rs = check_conv(ctx, p, pos, feat, n, row_ptr, col_idx, n_edges, out);
  if (rs != E2F_OK) return rs;
  hipStream_t s = (hipStream_t)stream;
  DeviceGuard g(ctx->device);
  const int L = p->lmax, C = p->channels, nk = nk_of(L);
  const e2f_ctx::CoefSet* cs = nullptr;
  if ((rs = coef_of(ctx, L, path_weights(p), true, cs)) != E2F_OK) return rs;
  if (n == 0) return E2F_OK;
  if (n_edges == 0) {
    E2F_HIP(launch_fill(out, (int64_t)n * nk * C, 0.0f, s));
    return E2F_OK;
  }
  const bool mixing = p->mix_w != nullptr;
  float* y = out;
  if (mixing) {
    rs = ensure(ctx, ctx->c, sizeof(float) * (size_t)n * nk * C, s);
    if (rs != E2F_OK) return rs;
    y = (float*)ctx->c.p;
  }
  E2F_TIMED("edge_tp", launch_edge_tp(with_coef(ctx, L, *cs), pos, feat, row_ptr, col_idx, alpha, n, n_edges, C,
                                      p->heads, y, s, p->y_norm != 0));
  if (mixing) E2F_TIMED("mix", launch_mix(L, y, p->mix_w, p->mix_dtype == E2F_BF16, n, C, out, s));
  return E2F_OK;
}

e2f_status e2f_wigner6j_conv_backward(e2f_ctx* ctx, const e2f_conv_params* p, const float* pos,
                                      const int32_t* graph_id, const float* feat, const float* grad_out, int32_t n,
                                      const int64_t* row_ptr, const int32_t* col_idx, int64_t n_edges,
                                      const float* alpha, float* grad_feat, float* grad_alpha, float* grad_pos,
                                      void* stream) {
  if (!grad_feat && !grad_alpha && !grad_pos) return fail(E2F_EINVAL, "no gradient is requested");
  if ((grad_alpha || grad_pos) && n > 0 && !feat) return fail(E2F_EINVAL, "feat is required for grad_alpha and grad_pos");
  e2f_status rs = check_params(ctx, p);
  if (rs != E2F_OK) return rs;
  if (p->y_norm) return fail(E2F_EUNSUPPORTED, "y_norm: the backward covers the plain layer only");
  if ((grad_alpha || grad_pos) && p->channels > 256)
    return fail(E2F_EUNSUPPORTED, "grad_alpha and grad_pos need channels <= 256");
  rs = check_conv(ctx, p, pos, grad_out, n, row_ptr, col_idx, n_edges, const_cast<float*>(grad_out));
  if (rs != E2F_OK) return rs;
  hipStream_t s = (hipStream_t)stream;
  DeviceGuard g(ctx->device);
  const int L = p->lmax, C = p->channels, H = p->heads, nk = nk_of(L), L1 = L + 1;
  const std::vector<double> w = path_weights(p);
  const e2f_ctx::CoefSet* cs = nullptr;
  if ((rs = coef_of(ctx, L, w, true, cs)) != E2F_OK) return rs;
  const DevTables tw = with_coef(ctx, L, *cs);
  if (n == 0) return E2F_OK;
  const bool mixing = p->mix_w != nullptr;
  const size_t wt_bytes = (size_t)L1 * C * C * (p->mix_dtype == E2F_BF16 ? 2 : 4);
  const size_t tmp_b = transpose_tmp_bytes(n, n_edges);
  const bool want_t = (grad_feat != nullptr || grad_pos != nullptr) && n_edges > 0;
  // the forces read the harmonic gradients of every edge from a table when it
  // stays under 4 GiB (else the per-edge kernel evaluates them itself)
  const size_t gt_bytes_full = sizeof(float) * 3 * (size_t)n_edges * nk;
  const char* gt_env = getenv("E2F_GEOM_GT");  // "0": always evaluate in the per-edge kernel (read per call)
  const size_t gt_bytes = grad_pos && n_edges > 0 && gt_bytes_full <= ((size_t)4 << 30) && !(gt_env && atoi(gt_env) == 0)
                              ? gt_bytes_full
                              : 0;
  const size_t need = (mixing ? al256(sizeof(float) * (size_t)n * nk * C) + al256(wt_bytes) : 0) +
                      (want_t ? 5 * al256(sizeof(int32_t) * (size_t)n_edges) + 2 * al256(sizeof(int64_t) * (n + 1)) +
                                    al256(sizeof(float) * (size_t)n_edges * H) + al256(tmp_b)
                              : 0) +
                      (grad_pos ? al256(sizeof(float) * (size_t)n_edges * 3) : 0) + al256(gt_bytes) + 256;
  rs = ensure(ctx, ctx->d, need, s);
  if (rs != E2F_OK) return rs;
  Carver cd{(char*)ctx->d.p};
  // ---- gradient of the unmixed output: y-bar = W^T out-bar per degree
  const float* gy = grad_out;
  if (mixing) {
    float* gyb = cd.take<float>((size_t)n * nk * C);
    void* WT = cd.take<char>(wt_bytes);
    E2F_TIMED("mix", launch_transpose_mix(p->mix_w, p->mix_dtype == E2F_BF16, L, C, WT, s));
    E2F_TIMED("mix", launch_mix(L, grad_out, WT, p->mix_dtype == E2F_BF16, n, C, gyb, s));
    gy = gyb;
  }
  if (n_edges == 0) {
    if (grad_pos) E2F_HIP(hipMemsetAsync(grad_pos, 0, sizeof(float) * (size_t)n * 3, s));
    if (grad_feat) E2F_HIP(hipMemsetAsync(grad_feat, 0, sizeof(float) * (size_t)n * nk * C, s));
    return E2F_OK;
  }
  // ---- the transposed graph (senders' rows), for the features and the positions
  int32_t* perm = nullptr;
  int32_t* colT = nullptr;
  int64_t* rowT = nullptr;
  float* alphaT = nullptr;
  int32_t* rows = nullptr;  // the receiver of every edge
  if (want_t) {
    rows = cd.take<int32_t>((size_t)n_edges);
    int32_t* iota = cd.take<int32_t>((size_t)n_edges);
    int32_t* keys_out = cd.take<int32_t>((size_t)n_edges);
    perm = cd.take<int32_t>((size_t)n_edges);
    colT = cd.take<int32_t>((size_t)n_edges);
    int64_t* cnt = cd.take<int64_t>((size_t)n + 1);
    rowT = cd.take<int64_t>((size_t)n + 1);
    alphaT = cd.take<float>((size_t)n_edges * H);
    void* tmp = cd.take<char>(tmp_b);
    E2F_TIMED("transpose", launch_transpose_graph(row_ptr, col_idx, alpha, n, n_edges, H, rows, iota, keys_out, perm,
                                                  cnt, rowT, colT, alpha ? alphaT : nullptr, tmp, tmp_b, s));
  }
  // ---- attention weights and positions: per edge, both from one product per
  // (receiver, head); then per atom the forces received minus those sent
  float* gedge = grad_pos ? cd.take<float>((size_t)n_edges * 3) : nullptr;
  float* Gt = gt_bytes ? cd.take<float>(gt_bytes / sizeof(float)) : nullptr;
  if (Gt) E2F_TIMED("edge_geom", launch_edge_shgrad(tw, pos, rows, col_idx, n_edges, Gt, s));
  if (grad_alpha || gedge) {
    const e2f_ctx::Geom* gsch = nullptr;
    if ((rs = geom_of(ctx, L, C / H, gsch)) != E2F_OK) return rs;
    E2F_TIMED("edge_geom", launch_edge_geom(tw, pos, feat, gy, row_ptr, col_idx, alpha, n, C, H, gsch->qc,
                                            gsch->meta, gsch->unit, gsch->oc, gsch->tot, Gt, n_edges, grad_alpha,
                                            gedge, s));
  }
  if (gedge) E2F_TIMED("force_gather", launch_force_gather(row_ptr, rowT, perm, gedge, n, grad_pos, s));
  // ---- features: the same layer on the transposed graph, input degree o,
  // output degree a, weights w[a][f][o] kappa(a,f,o) (-1)^f
  if (grad_feat) {
    const std::vector<double>* kap = nullptr;
    rs = transpose_factors(ctx, L, kap);
    if (rs != E2F_OK) return rs;
    std::vector<double> wt((size_t)L1 * L1 * L1, 0.0);
    for (int a = 0; a <= L; ++a)
      for (int f = 0; f <= L; ++f)
        for (int o = std::abs(a - f); o <= std::min(a + f, L); ++o) {
          const size_t q = ((size_t)a * L1 + f) * L1 + o;
          wt[((size_t)o * L1 + f) * L1 + a] = w[q] * (*kap)[q] * ((f & 1) ? -1.0 : 1.0);
        }
    e2f_conv_params pt = *p;
    pt.path_w = wt.data();
    pt.mix_w = nullptr;
    // the forward on the transposed graph, in a workspace of the context's
    // own (the backward's buffers, which it reads, stay where they are)
    const size_t fb = fwd_layout(&pt, n, n_edges, alpha != nullptr).total(n);
    if ((rs = ensure(ctx, ctx->c, fb, s)) != E2F_OK) return rs;
    return forward_impl(ctx, &pt, pos, graph_id, gy, n, rowT, colT, n_edges, alpha ? alphaT : nullptr, grad_feat,
                        ctx->c.p, ctx->c.n, stream, true);
  }
  return E2F_OK;
}

e2f_status e2f_wigner6j_conv_forward_dense(e2f_ctx* ctx, const e2f_conv_params* p, const float* pos,
                                           const float* feat, int32_t n, const float* alpha, float* out,
                                           void* stream) {
  e2f_status rs = check_params(ctx, p);
  if (rs != E2F_OK) return rs;
  if (n < 0) return fail(E2F_EINVAL, "n < 0");
  if (n > 0 && (!pos || !feat || !out)) return fail(E2F_EINVAL, "pos, feat and out are required");
  if ((double)n * n * p->heads > 4.0e9) return fail(E2F_EUNSUPPORTED, "N^2 H = %.3g attention weights", (double)n * n * p->heads);
  if (p->y_norm) return fail(E2F_EUNSUPPORTED, "y_norm: not available on this entry point");
  if (ctx->device < 0) return fail(E2F_EDEVICE, "context has no device");
  hipStream_t s = (hipStream_t)stream;
  DeviceGuard g(ctx->device);
  const int L = p->lmax, C = p->channels, H = p->heads, nk = nk_of(L), dh = C / H;
  const e2f_ctx::CoefSet* cs = nullptr;
  if ((rs = coef_of(ctx, L, path_weights(p), true, cs)) != E2F_OK) return rs;
  if (n == 0) return E2F_OK;
  const DevTables t = with_coef(ctx, L, *cs);
  const size_t rowb = sizeof(float) * (size_t)t.dimT * C;
  const bool mixing = p->mix_w != nullptr;
  const size_t need = al256(sizeof(int) * 16) + al256(sizeof(double) * 3) + al256(sizeof(double) * (size_t)n * nk) +
                      2 * al256(rowb * (size_t)n) + al256(sizeof(float) * (size_t)n * dense_lda(n) * H) +
                      al256(sizeof(int32_t) * (size_t)n) + (mixing ? al256(sizeof(float) * (size_t)n * nk * C) : 0);
  rs = ensure(ctx, ctx->b, need, s);
  if (rs != E2F_OK) return rs;
  Carver cb{(char*)ctx->b.p};
  int* stats = cb.take<int>(16);
  double* org = cb.take<double>(3);
  double* R = cb.take<double>((size_t)n * nk);
  float* T = cb.take<float>((size_t)n * t.dimT * C);
  float* S = cb.take<float>((size_t)n * t.dimT * C);
  float* A = cb.take<float>((size_t)n * dense_lda(n) * H);
  int32_t* order = cb.take<int32_t>((size_t)n);
  float* y = mixing ? cb.take<float>((size_t)n * nk * C) : out;
  // one origin, the centre of the bounding box (the products couple every
  // pair), found on the device
  E2F_TIMED("bbox", launch_plan_bbox(pos, nullptr, n, stats, nullptr, s));
  E2F_TIMED("bbox", launch_plan_centre(stats, org, s));
  E2F_TIMED("sh", launch_sh(t, pos, nullptr, org, nullptr, nullptr, 1, n, R, nullptr, s));
  E2F_TIMED("node_tp", launch_node_tp(t, R, nullptr, feat, n, C, dh, T, s));
  E2F_TIMED("tile_plan", launch_dense_alpha(alpha, n, H, A, s));
  E2F_TIMED("tile_plan", launch_iota(n, order, s));
  E2F_TIMED("aggregate", launch_dense_aggregate(A, n, T, t.dimT, C, H, S, s));
  E2F_TIMED("recouple", launch_recouple(t, R, S, false, order, n, C, dh, y, s));
  if (mixing) E2F_TIMED("mix", launch_mix(L, y, p->mix_w, p->mix_dtype == E2F_BF16, n, C, out, s));
  return E2F_OK;
}

e2f_status e2f_wigner6j_conv_forward_global(e2f_ctx* ctx, const e2f_conv_params* p, const float* pos,
                                            const float* feat, int32_t n, float* out, void* stream) {
  e2f_status rs = check_params(ctx, p);
  if (rs != E2F_OK) return rs;
  if (n < 0) return fail(E2F_EINVAL, "n < 0");
  if (n > 0 && (!pos || !feat || !out)) return fail(E2F_EINVAL, "pos, feat and out are required");
  if (p->y_norm) return fail(E2F_EUNSUPPORTED, "y_norm: not available on this entry point");
  if (ctx->device < 0) return fail(E2F_EDEVICE, "context has no device");
  hipStream_t s = (hipStream_t)stream;
  DeviceGuard g(ctx->device);
  const int L = p->lmax, C = p->channels, nk = nk_of(L), dh = C / p->heads;
  const e2f_ctx::CoefSet* cs = nullptr;
  if ((rs = coef_of(ctx, L, path_weights(p), true, cs)) != E2F_OK) return rs;
  if (n == 0) return E2F_OK;
  const DevTables t = with_coef(ctx, L, *cs);
  // the moment of the uncoupled products G[be][(q, c)] = sum_j R_be(p_j) h_j[q][c]
  // (fp64, fixed order), coupled once into the shared S row
  const int64_t W = (int64_t)t.dimT * C, WG = (int64_t)nk * nk * C;
  const int G = global_groups(n, nk, C);
  const bool mixing = p->mix_w != nullptr;
  const size_t need = al256(sizeof(int) * 16) + al256(sizeof(double) * 3) + al256(sizeof(double) * (size_t)n * nk) +
                      al256(sizeof(double) * (size_t)G * WG) + al256(sizeof(double) * (size_t)WG) +
                      al256(sizeof(float) * (size_t)W) + al256(sizeof(int32_t) * (size_t)n) +
                      (mixing ? al256(sizeof(float) * (size_t)n * nk * C) : 0);
  rs = ensure(ctx, ctx->b, need, s);
  if (rs != E2F_OK) return rs;
  Carver cb{(char*)ctx->b.p};
  int* stats = cb.take<int>(16);
  double* org = cb.take<double>(3);
  double* R = cb.take<double>((size_t)n * nk);
  double* part = cb.take<double>((size_t)G * WG);
  double* G64 = cb.take<double>((size_t)WG);
  float* M32 = cb.take<float>((size_t)W);
  int32_t* order = cb.take<int32_t>((size_t)n);
  float* y = mixing ? cb.take<float>((size_t)n * nk * C) : out;
  // one origin, the centre of the bounding box (every pair is coupled), found on the device
  E2F_TIMED("bbox", launch_plan_bbox(pos, nullptr, n, stats, nullptr, s));
  E2F_TIMED("bbox", launch_plan_centre(stats, org, s));
  E2F_TIMED("sh", launch_sh(t, pos, nullptr, org, nullptr, nullptr, 1, n, R, nullptr, s));
  E2F_TIMED("aggregate", launch_global_moment(t, R, feat, n, C, dh, part, G64, M32, s));
  E2F_TIMED("tile_plan", launch_iota(n, order, s));
  E2F_TIMED("recouple", launch_recouple(t, R, M32, true, order, n, C, dh, y, s));
  if (mixing) E2F_TIMED("mix", launch_mix(L, y, p->mix_w, p->mix_dtype == E2F_BF16, n, C, out, s));
  return E2F_OK;
}

e2f_status e2f_last_slices(const e2f_ctx* ctx, int64_t* slices) {
  if (!ctx || !slices) return fail(E2F_EINVAL, "ctx and slices are required");
  *slices = ctx->last_slices;
  return E2F_OK;
}

e2f_status e2f_profile(e2f_ctx* ctx, int enable) {
  if (!ctx) return fail(E2F_EINVAL, "ctx is NULL");
  if (ctx->device < 0) return fail(E2F_EDEVICE, "context has no device");
  DeviceGuard g(ctx->device);
  E2F_HIP(hipDeviceSynchronize());
  for (auto& r : ctx->recs) {
    ctx->pool.push_back(r.start);
    ctx->pool.push_back(r.stop);
  }
  ctx->recs.clear();
  ctx->prof = enable != 0;
  return E2F_OK;
}

e2f_status e2f_profile_read(e2f_ctx* ctx, char* buf, size_t bytes) {
  if (!ctx || !buf || bytes == 0) return fail(E2F_EINVAL, "ctx and buf are required");
  if (ctx->device < 0) return fail(E2F_EDEVICE, "context has no device");
  DeviceGuard g(ctx->device);
  std::vector<std::string> names;
  std::vector<double> ms;
  std::vector<long> cnt;
  for (auto& r : ctx->recs) {
    E2F_HIP(hipEventSynchronize(r.stop));
    float t = 0.0f;
    E2F_HIP(hipEventElapsedTime(&t, r.start, r.stop));
    size_t k = 0;
    while (k < names.size() && names[k] != r.name) ++k;
    if (k == names.size()) {
      names.emplace_back(r.name);
      ms.push_back(0.0);
      cnt.push_back(0);
    }
    ms[k] += t;
    cnt[k] += 1;
  }
  std::string out;
  char line[128];
  for (size_t k = 0; k < names.size(); ++k) {
    snprintf(line, sizeof(line), "%s %ld %.6f\n", names[k].c_str(), cnt[k], ms[k]);
    out += line;
  }
  if (out.size() + 1 > bytes) return fail(E2F_ECAPACITY, "profile text needs %zu bytes", out.size() + 1);
  std::memcpy(buf, out.c_str(), out.size() + 1);
  return E2F_OK;
}

}  // extern "C"
