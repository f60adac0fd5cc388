"""ckks_linear_mac_scalar_noalloc against ckks_linear_mac_scalar, through the C ABI.

The no-allocation entry point takes the matrix-core workspace from the
library's own per-GPU scratch array.  Two calls in a row, the second with a
smaller layer (so the scratch still holds the first call's fragments), must
each equal the workspace entry point's output bit for bit (and the oracle's on
sampled rows); a request whose workspace exceeds the array is refused."""
import numpy as np
import pytest

from oracle import encode as OE
from oracle import linear as OL
from workloads import gen

pytestmark = pytest.mark.gpu


def _layer(ck, ctx, d_out, d_in, seed):
    qs, L, n = ctx.moduli, ctx.limbs, ctx.n
    rng = np.random.default_rng(seed)
    W = gen.scalar_weights(rng, d_out, d_in)
    ct = gen.uniform_residues(rng, (d_in, 2), qs, n)
    w_enc = OE.encode_scalar(W, 2.0 ** 26, qs).astype(np.uint32)
    return w_enc, ct


def _both(ck, ctx, w_enc, ct, d_out, d_in):
    L, n = ctx.limbs, ctx.n
    d_w, d_ct = ck.to_device(w_enc), ck.to_device(ct)
    ws = ck.empty_u32((ck.ckks_workspace_bytes(ctx, ck.CKKS_OP_MAC_SCALAR, d_out, d_in, L) // 4 + 4,))
    ref = ck.empty_u32((d_out, 2, L, n))
    ck.ckks_linear_mac_scalar(ctx, d_w, d_ct, ref, d_out, d_in, L, ws)
    got = ck.empty_u32((d_out, 2, L, n))
    got.fill_(-1)
    ck.ckks_linear_mac_scalar_noalloc(ctx, d_w, d_ct, got, d_out, d_in, L)
    return ck.to_host_u32(ref), ck.to_host_u32(got)


def test_noalloc_mac_matches_the_workspace_entry_point(gpu_lib):
    ck = gpu_lib
    ctx = ck.Context(12, 3)
    assert ck.ckks_workspace_bytes(ctx, ck.CKKS_OP_MAC_SCALAR, 300, 200, 3) <= ck.NOALLOC_SCRATCH_BYTES
    # first call: 300 x 200 (3 row tiles, the last ragged; 4 k-steps, the last ragged)
    w1, c1 = _layer(ck, ctx, 300, 200, 9001)
    ref1, got1 = _both(ck, ctx, w1, c1, 300, 200)
    assert np.array_equal(got1, ref1)
    rows = [0, 137, 299]
    want = OL.mac_scalar(w1, c1, ctx.moduli, rows=rows)
    assert np.array_equal(got1[rows], want.astype(np.uint32))
    # second call, smaller (40 x 70): the scratch still holds the first call's fragments
    w2, c2 = _layer(ck, ctx, 40, 70, 9002)
    ref2, got2 = _both(ck, ctx, w2, c2, 40, 70)
    assert np.array_equal(got2, ref2)
    assert np.array_equal(got2[[0, 39]], OL.mac_scalar(w2, c2, ctx.moduli, rows=[0, 39]).astype(np.uint32))
    ctx.close()


def test_noalloc_mac_refuses_requests_beyond_its_scratch(gpu_lib):
    ck = gpu_lib
    ctx = ck.Context(10, 4)
    d_out, d_in, L = 1200, 4096, 4
    need = ck.ckks_workspace_bytes(ctx, ck.CKKS_OP_MAC_SCALAR, d_out, d_in, L)
    assert need > ck.NOALLOC_SCRATCH_BYTES
    w = ck.empty_u32((d_out, d_in, L))
    ct = ck.empty_u32((d_in, 2, L, ctx.n))
    out = ck.empty_u32((d_out, 2, L, ctx.n))
    with pytest.raises(ck.CkksError) as e:
        ck.ckks_linear_mac_scalar_noalloc(ctx, w, ct, out, d_out, d_in, L)
    assert e.value.code == ck.CKKS_E_WORKSPACE
    assert "scratch" in str(e.value)
    ctx.close()


def test_noalloc_mac_replays_under_graph_capture(gpu_lib):
    """The caller the entry point is for: a HIP graph captures the call (it allocates
    nothing and records no memset) and is replayed three times, with eager work
    of the program's own between the replays (a workspace MAC on other inputs, the
    scratch's other user); every replay equals the eager result."""
    import torch
    ck = gpu_lib
    ctx = ck.Context(11, 3)
    L, n = ctx.limbs, ctx.n
    w1, c1 = _layer(ck, ctx, 130, 96, 9003)
    w2, c2 = _layer(ck, ctx, 64, 64, 9004)
    d_w1, d_c1 = ck.to_device(w1), ck.to_device(c1)
    d_w2, d_c2 = ck.to_device(w2), ck.to_device(c2)
    out = ck.empty_u32((130, 2, L, n))
    eager = ck.empty_u32((130, 2, L, n))
    ck.ckks_linear_mac_scalar_noalloc(ctx, d_w1, d_c1, eager, 130, 96, L)
    other = ck.empty_u32((64, 2, L, n))
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        ck.ckks_linear_mac_scalar_noalloc(ctx, d_w1, d_c1, out, 130, 96, L, stream=s)   # warm-up on the stream
    s.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        ck.ckks_linear_mac_scalar_noalloc(ctx, d_w1, d_c1, out, 130, 96, L, stream=s)
    for k in range(3):
        out.fill_(0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {k}"
        ck.ckks_linear_mac_scalar_noalloc(ctx, d_w2, d_c2, other, 64, 64, L)           # eager use of the scratch
        torch.cuda.synchronize()
    assert np.array_equal(ck.to_host_u32(other)[[0, 63]],
                          OL.mac_scalar(w2, c2, ctx.moduli, rows=[0, 63]).astype(np.uint32))
    del g
    ctx.close()
