"""The forward for callers that cannot allocate: the scratch-memory entry
point against the workspace entry point, on two calls in a row (the second
with a smaller input, so stale scratch contents from the first are present),
through the C ABI.  Run with -m gpu."""
import numpy as np
import pytest
import torch

import e2f_synth as syn
import oracle as o
from cases import TOL_F32, case

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def gpu(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def test_forward_without_allocation():
    import paper_2501_19216_amd as e2f
    ctx = e2f.e2f_create(4, 0)
    try:
        runs = []
        for name in ("molecules256x30_L3", "cluster32_L2"):  # the second input is smaller
            inp, rp, ci, alpha = case(name)
            wl = inp.workload
            args = (gpu(inp.pos), gpu(inp.feat), gpu(rp), gpu(ci), gpu(alpha), wl.lmax, wl.heads, wl.cutoff)
            kw = dict(mix_w=gpu(inp.mix_w), graph_id=gpu(inp.graph_id))
            print("no-alloc forward: %s, %d atoms, %d edges" % (name, inp.pos.shape[0], len(ci)), flush=True)
            if not runs:
                # parameters not yet resident: refused without any device work
                with pytest.raises(e2f.E2FError) as ei:
                    e2f.e2f_wigner6j_conv_forward_noalloc(ctx, *args, **kw)
                assert ei.value.status == e2f.E2F_EINVAL
            e2f.e2f_wigner6j_prepare(ctx, wl.lmax, wl.channels, wl.heads, wl.cutoff, mix_w=kw["mix_w"])
            out = torch.full_like(gpu(inp.feat), float("nan"))
            e2f.e2f_wigner6j_conv_forward_noalloc(ctx, *args, **kw, out=out)
            want = e2f.e2f_wigner6j_conv_forward(ctx, *args, **kw)
            got = out.cpu().numpy()
            ref = want.cpu().numpy()
            assert np.isfinite(got).all()
            err = o.max_rel_err(got, ref.astype(np.float64), wl.lmax)
            print("no-alloc forward: %s err vs workspace entry %.3e" % (name, err), flush=True)
            assert err <= TOL_F32
            runs.append(name)
        # the fused form (split-bf16 products, F_i per receiver, re-laid
        # features) in the scratch memory, after the two-kernel calls above
        inp, rp, ci, alpha = case("water2000_L4")
        wl = inp.workload
        args = (gpu(inp.pos), gpu(inp.feat), gpu(rp), gpu(ci), gpu(alpha), wl.lmax, wl.heads, wl.cutoff)
        print("no-alloc forward: water2000_L4 fused, %d atoms, %d edges" % (inp.pos.shape[0], len(ci)), flush=True)
        e2f.e2f_wigner6j_prepare(ctx, wl.lmax, wl.channels, wl.heads, wl.cutoff, form="fused")
        out = torch.full_like(gpu(inp.feat), float("nan"))
        e2f.e2f_wigner6j_conv_forward_noalloc(ctx, *args, out=out, form="fused")
        want = e2f.e2f_wigner6j_conv_forward(ctx, *args, form="fused").cpu().numpy()
        got = out.cpu().numpy()
        assert np.isfinite(got).all()
        err = o.max_rel_err(got, want.astype(np.float64), wl.lmax)
        print("no-alloc forward: water2000_L4 fused err vs workspace entry %.3e" % err, flush=True)
        assert err <= TOL_F32
        # an input whose smallest workspace exceeds the scratch memory
        inp, rp, ci, alpha = case("protein20k_L4")
        wl = inp.workload
        e2f.e2f_wigner6j_prepare(ctx, wl.lmax, wl.channels, wl.heads, wl.cutoff)
        with pytest.raises(e2f.E2FError) as ei:
            e2f.e2f_wigner6j_conv_forward_noalloc(ctx, gpu(inp.pos), gpu(inp.feat), gpu(rp), gpu(ci), gpu(alpha),
                                                  wl.lmax, wl.heads, wl.cutoff)
        assert ei.value.status == e2f.E2F_ECAPACITY
    finally:
        ctx.close()
