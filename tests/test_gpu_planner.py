"""GPU execution of residency plans (section 3.3's pin / fallback-encode and
refresh lines): the result does not depend on the budget, and the chain equals
the oracle's composition of encode_poly, mac_poly, rescale and refresh."""
import numpy as np
import pytest

from oracle import encode as OE
from oracle import linear as OL
from oracle import rlwe as OR
from paper_2606_17421_amd.planner import Executor, LinearGroup, plan
from workloads import gen

pytestmark = pytest.mark.gpu

LOG_N, L, SCALE = 10, 4, float(1 << 25)


def model(d, layers):
    return [LinearGroup(f"g{i}", d, d, tee_after=(i == 1)) for i in range(layers)]


def secret_inputs(ck, ctx, d, seed, refreshes):
    """Secret (host and NTT form on the device), one fresh (a, e) draw per refresh
    (host arrays and device tensors) and the input ciphertexts."""
    qs, n = ctx.moduli, ctx.n
    st = gen.streams(seed, LOG_N)
    s = gen.ternary_secret(st["secret"], n)
    s_res = np.stack([np.mod(s, q) for q in qs]).astype(np.uint32)
    s_ntt = ck.to_device(s_res)
    ck.ckks_ntt(ctx, s_ntt, 1, L)
    draws = [(gen.uniform_residues(st["residues"], (d,), qs, n), gen.gaussian_error(st["error"], (d, n)).astype(np.int32))
             for _ in range(refreshes)]
    ct = gen.uniform_residues(st["residues"], (d, 2), qs, n)
    return s, s_ntt, draws, [(ck.to_device(a), ck.to_device(e)) for a, e in draws], ct


def run(ck, ctx, groups, budget, weights_dev, s_ntt, draws_dev, ct_dev):
    p = plan(groups, budget, L, ctx.n)
    ex = Executor(ctx, p, weights_dev, SCALE, s_ntt)
    out, limbs = ex.run(ct_dev, draws_dev)
    d = groups[-1].d_out
    return p, ck.to_host_u32(out[: d * 2 * limbs * ctx.n]).reshape(d, 2, limbs, ctx.n)


def test_result_does_not_depend_on_the_budget(gpu_lib):
    ck = gpu_lib
    ctx = ck.Context(LOG_N, L)
    d, layers = 8, 5
    groups = model(d, layers)
    st = gen.streams(501, LOG_N)
    W = [gen.poly_weights(st["weights"], d, d, ctx.n // 2).reshape(d * d, ctx.n // 2) for _ in range(layers)]
    Wd = [ck.to_device(np.ascontiguousarray(w)) for w in W]
    full = plan(groups, 1 << 40, L, ctx.n)
    s, s_ntt, draws, draws_dev, ct = secret_inputs(ck, ctx, d, 502, full.refreshes)
    ct_dev = ck.to_device(ct)
    outs = {}
    for budget in (1 << 40, 0, full.steps[0].encoded_bytes + full.steps[1].encoded_bytes):
        p, outs[budget] = run(ck, ctx, groups, budget, Wd, s_ntt, draws_dev, ct_dev)
        assert p.pinned + p.fallback == layers
    ref = outs[1 << 40]
    for budget, o in outs.items():
        assert np.array_equal(o, ref), budget
    assert plan(groups, 0, L, ctx.n).fallback == layers


def test_executor_refuses_reused_refresh_randomness(gpu_lib):
    """Every refresh of a pass takes its own (a, e): too few draws, or two draws that
    share storage, are refused before anything runs."""
    import pytest as _pt
    ck = gpu_lib
    ctx = ck.Context(LOG_N, L)
    d, layers = 4, 5
    groups = model(d, layers)
    p = plan(groups, 1 << 40, L, ctx.n)
    assert p.refreshes >= 2
    rng = np.random.default_rng(507)
    W = [ck.to_device(gen.poly_weights(rng, d, d, ctx.n // 2).reshape(d * d, ctx.n // 2)) for _ in range(layers)]
    s, s_ntt, draws, draws_dev, ct = secret_inputs(ck, ctx, d, 508, p.refreshes)
    ex = Executor(ctx, p, W, SCALE, s_ntt)
    with _pt.raises(ValueError):
        ex.run(ck.to_device(ct), draws_dev[:-1])
    with _pt.raises(ValueError):
        ex.run(ck.to_device(ct), [draws_dev[0]] * p.refreshes)
    ex.run(ck.to_device(ct), draws_dev)


def test_chain_equals_the_oracle_composition(gpu_lib):
    """Constant-slot weights encode exactly on both sides (the constant polynomial
    round(c scale)), so the GPU chain is compared with the oracle bit for bit."""
    ck = gpu_lib
    ctx = ck.Context(LOG_N, L)
    qs, psis, n = ctx.moduli, ctx.roots, ctx.n
    d, layers = 4, 5                       # two refreshes: after the TEE window and when the level runs out
    groups = model(d, layers)
    rng = np.random.default_rng(503)
    consts = [rng.normal(0, 0.02, (d, d)) for _ in range(layers)]
    W = [np.repeat(c.reshape(d * d, 1), n // 2, axis=1) for c in consts]
    refreshes = plan(groups, 1 << 40, L, n).refreshes
    assert refreshes >= 2
    s, s_ntt, draws, draws_dev, ct = secret_inputs(ck, ctx, d, 504, refreshes)
    p, got = run(ck, ctx, groups, 1 << 40, [ck.to_device(w) for w in W], s_ntt, draws_dev, ck.to_device(ct))
    cur = ct.astype(np.uint64)
    it = iter(draws)
    for step, w in zip(p.steps, W):
        lv = step.level
        pt = OE.encode_poly(w.reshape(d, d, n // 2), SCALE, qs[:lv], psis[:lv], LOG_N)
        mac = OL.mac_poly(pt, cur, qs[:lv])
        cur = OL.rescale(mac, qs[:lv], psis[:lv], LOG_N)
        if step.refresh_after:
            a, e = next(it)
            cur = OR.refresh(cur, s, a, e, qs, psis, LOG_N, L)
    assert got.shape == cur.shape
    assert np.array_equal(got, cur.astype(np.uint32))


def test_chain_at_the_benchmarked_width(gpu_lib):
    """Three groups of the benchmarked stack's width (32 x 32, N = 2^14, 4 limbs, a TEE
    window after the first), one pinned and two fallback, against the oracle's chain.
    Constant-slot weights: the NTT form of the constant polynomial round(c scale) is that
    constant in every slot, so the oracle's plaintexts are its scalar encodings (the
    equality of the two encodings for constant slots is pinned on the oracle side)."""
    ck = gpu_lib
    log_n, L, d = 14, 4, 32
    ctx = ck.Context(log_n, L)
    qs, psis, n = ctx.moduli, ctx.roots, ctx.n
    groups = [LinearGroup(f"g{i}", d, d, tee_after=(i == 0)) for i in range(3)]
    rng = np.random.default_rng(505)
    consts = [rng.normal(0, 0.02, (d, d)) for _ in groups]
    W = [np.repeat(c.reshape(d * d, 1), n // 2, axis=1) for c in consts]
    st = gen.streams(506, log_n)
    s = gen.ternary_secret(st["secret"], n)
    s_res = np.stack([np.mod(s, q) for q in qs]).astype(np.uint32)
    s_ntt = ck.to_device(s_res)
    ck.ckks_ntt(ctx, s_ntt, 1, L)
    budget = plan(groups, 1 << 40, L, n).steps[0].encoded_bytes           # only the first group fits
    p = plan(groups, budget, L, n)
    assert [st_.pinned for st_ in p.steps] == [True, False, False]
    draws = [(gen.uniform_residues(st["residues"], (d,), qs, n), gen.gaussian_error(st["error"], (d, n)).astype(np.int32))
             for _ in range(p.refreshes)]
    ct = gen.uniform_residues(st["residues"], (d, 2), qs, n)
    ex = Executor(ctx, p, [ck.to_device(w) for w in W], SCALE, s_ntt)
    out, limbs = ex.run(ck.to_device(ct), [(ck.to_device(a), ck.to_device(e)) for a, e in draws])
    got = ck.to_host_u32(out[: d * 2 * limbs * n]).reshape(d, 2, limbs, n)
    cur = ct.astype(np.uint64)
    for step, c in zip(p.steps, consts):
        lv = step.level
        w_enc = OE.encode_scalar(c, SCALE, qs[:lv])                              # (d, d, lv)
        pt = np.broadcast_to(w_enc[..., None], (d, d, lv, n))
        cur = OL.rescale(OL.mac_poly(pt, cur, qs[:lv]), qs[:lv], psis[:lv], log_n)
        if step.refresh_after:
            a, e = draws[sum(x.refresh_after for x in p.steps[: p.steps.index(step)])]
            cur = OR.refresh(cur, s, a, e, qs, psis, log_n, L)
    assert np.array_equal(got, cur.astype(np.uint32))
