"""Encoded-weight residency planning and plan execution for a stack of
full-polynomial linear groups (the pin / fallback-encode lines of the paper's
boundary-aware scheduler, Algorithm 1 in section 3.3, and the persistent
versus fallback-encode modes of section 4.2).

`plan()` walks the linear groups in topological order with a device budget
for encoded weights: a group whose NTT-form plaintexts fit the remaining
budget is pinned (encoded once, kept resident), otherwise it is re-encoded on
every call (fallback).  It also tracks the ciphertext level: every group is a
ct x pt MAC followed by a rescale (one limb dropped), and a decrypt-then-
encrypt refresh back to the full chain is inserted after a group when a TEE
window follows it or when the next group's output would keep fewer than two
limbs (the refresh decrypts with limbs 0 and 1).

`Executor` runs a plan through the C ABI (encode_poly, mac_poly, rescale,
refresh): pinned plaintexts are encoded at set-up at the level their group
runs at; fallback groups keep their slot vectors on the device and encode into
one shared plaintext buffer per call.  Results do not depend on the plan, only
the time does.
"""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class LinearGroup:
    """One linear operator group: d_in ciphertexts in, d_out out, full-polynomial
    weights (d_out x d_in slot vectors).  tee_after: a TEE window (decrypt-compute-
    encrypt) follows the group, so its output is refreshed to the full chain."""
    name: str
    d_out: int
    d_in: int
    tee_after: bool = False


@dataclass(frozen=True)
class Step:
    group: LinearGroup
    level: int                 # limbs of the group's input ciphertexts
    pinned: bool               # encoded weights resident (else fallback encode per call)
    encoded_bytes: int         # NTT-form plaintext bytes at that level
    refresh_after: bool        # DtE refresh of the rescaled output back to the full chain


@dataclass
class Plan:
    steps: list[Step] = field(default_factory=list)
    budget_bytes: int = 0
    pinned_bytes: int = 0

    @property
    def pinned(self) -> int:
        return sum(s.pinned for s in self.steps)

    @property
    def fallback(self) -> int:
        return sum(not s.pinned for s in self.steps)

    @property
    def refreshes(self) -> int:
        return sum(s.refresh_after for s in self.steps)


def encoded_bytes(g: LinearGroup, level: int, n: int) -> int:
    return g.d_out * g.d_in * level * n * 4


def plan(groups, budget_bytes: int, full_limbs: int, n: int, min_out_limbs: int = 2) -> Plan:
    """Residency and level plan (section 3.3, Algorithm 1: pin / fallback encode,
    DtE refresh when the level budget runs out).

    full_limbs: limbs of a fresh (or refreshed) ciphertext.  min_out_limbs: the
    fewest limbs a group's rescaled output may keep (the refresh decrypts with
    limbs 0 and 1, so at least 2); a refresh follows a group whenever the next
    group's output would fall below it.
    """
    if min_out_limbs < 2 or full_limbs < min_out_limbs + 1:
        raise ValueError("the chain must allow one rescale that keeps min_out_limbs >= 2 limbs")
    groups = list(groups)
    for a, b in zip(groups, groups[1:]):
        if a.d_out != b.d_in:
            raise ValueError(f"{a.name} -> {b.name}: {a.d_out} outputs feed {b.d_in} inputs")
    p = Plan(budget_bytes=budget_bytes)
    left = budget_bytes
    level = full_limbs
    for i, g in enumerate(groups):
        size = encoded_bytes(g, level, n)
        pin = size <= left
        if pin:
            left -= size
            p.pinned_bytes += size
        after = level - 1                                  # the rescale drops one limb
        last = i + 1 == len(groups)
        refresh = not last and (g.tee_after or after - 1 < min_out_limbs)
        p.steps.append(Step(g, level, pin, size, refresh))
        level = full_limbs if refresh else after
    return p


def _span(t):
    """Byte range [start, end) of a tensor's storage view."""
    start = t.data_ptr()
    return start, start + t.numel() * t.element_size()


def check_refresh_draws(draws, needed: int) -> None:
    """The randomness of a pass's refreshes: at least `needed` (a, e) pairs, and no
    two pairs sharing storage.  A refresh is Enc(Dec(ct)) (section 3.2); encrypting
    two different plaintexts with the same (a, e) would hand the untrusted side the
    difference of the plaintexts (c0 - c0' = m - m'), so every refresh takes its own."""
    draws = list(draws)
    if len(draws) < needed:
        raise ValueError(f"the plan has {needed} refreshes but {len(draws)} (a, e) draws were given")
    spans = []
    for k, (a, e) in enumerate(draws[:needed]):
        for t in (a, e):
            lo, hi = _span(t)
            for lo2, hi2, k2 in spans:
                if lo < hi2 and lo2 < hi:
                    raise ValueError(f"refresh draws {k2} and {k} share storage: each refresh needs fresh (a, e)")
            spans.append((lo, hi, k))


class Executor:
    """Runs a Plan on the GPU through the library's entry points.

    weights: per group a cuda float64 tensor [d_out * d_in][N/2] of slot values
    (kept for fallback groups; pinned groups are encoded once here).
    s_ntt: the secret in NTT form, cuda [full_limbs][N] (the refreshes run on the
    trusted side of each boundary crossing).  The randomness of the refreshes is
    an argument of run(), drawn anew by the caller for every pass.
    """

    def __init__(self, ctx, the_plan: Plan, weights, scale: float, s_ntt, stream=None):
        import torch

        import paper_2606_17421_amd as ck
        self.ck, self.ctx, self.plan, self.scale, self.stream = ck, ctx, the_plan, scale, stream
        self.s_ntt = s_ntt
        n = ctx.n
        self.full_limbs = max(s.level for s in the_plan.steps)
        self.pts, self.slots = [], []
        fallback_bytes = 0
        for s, w in zip(the_plan.steps, weights):
            g = s.group
            if s.pinned:
                pt = ck.empty_u32((g.d_out, g.d_in, s.level, n), device=ctx.device)
                ck.ckks_linear_encode_poly(ctx, w, g.d_out * g.d_in, s.level, scale, pt, stream)
                self.pts.append(pt)
                self.slots.append(None)
            else:
                self.pts.append(None)
                self.slots.append(w)
                fallback_bytes = max(fallback_bytes, s.encoded_bytes)
        self.scratch_pt = (torch.empty((fallback_bytes // 4,), dtype=torch.int32, device=f"cuda:{ctx.device}")
                           if fallback_bytes else None)
        d_max = max(max(s.group.d_out, s.group.d_in) for s in the_plan.steps)
        self.buf = [ck.empty_u32((d_max * 2 * self.full_limbs * n,), device=ctx.device) for _ in range(3)]

    def run(self, ct_in, refresh_draws=(), events=None):
        """One pass over the plan.  ct_in: cuda [d_in][2][full_limbs][N].
        refresh_draws: one (a, e) pair per refresh of the plan, in plan order, each
        freshly drawn for this pass (a: cuda [d_out][full_limbs][N] uniform residues in
        NTT form; e: cuda int32 [d_out][N] error coefficients); pairs must not share
        storage.  Returns the output tensor (a view into an internal buffer,
        [d_out][2][limbs][N]) and its limbs.
        events: optional list; per step a (start, after_encode, end) triple of cuda events."""
        import torch
        ck, ctx, n, st = self.ck, self.ctx, self.ctx.n, self.stream
        check_refresh_draws(refresh_draws, self.plan.refreshes)
        draws = iter(refresh_draws)
        cur, limbs = ct_in, self.plan.steps[0].level
        # buffers: 0 = MAC output, 1 = rescale output, 2 = refresh output; a group's
        # input (1 or 2, or ct_in) is consumed by its MAC before 1 is rewritten
        for s, pt, w in zip(self.plan.steps, self.pts, self.slots):
            g = s.group
            assert limbs == s.level
            ev = None
            if events is not None:
                ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
                ev[0].record(st if st is not None else torch.cuda.current_stream())
            if pt is None:
                pt = self.scratch_pt[: g.d_out * g.d_in * limbs * n]
                ck.ckks_linear_encode_poly(ctx, w, g.d_out * g.d_in, limbs, self.scale, pt, st)
            if ev is not None:
                ev[1].record(st if st is not None else torch.cuda.current_stream())
            mac = self.buf[0][: g.d_out * 2 * limbs * n]
            res = self.buf[1][: g.d_out * 2 * (limbs - 1) * n]
            ck.ckks_linear_mac_poly(ctx, pt, cur, mac, g.d_out, g.d_in, limbs, st)
            ck.ckks_rescale(ctx, mac, res, g.d_out, limbs, None, stream=st)
            cur, limbs = res, limbs - 1
            if s.refresh_after:
                out = self.buf[2][: g.d_out * 2 * self.full_limbs * n]
                a, e = next(draws)
                ck.ckks_refresh(ctx, res, limbs, self.s_ntt, a, e, g.d_out, self.full_limbs, out, st)
                cur, limbs = out, self.full_limbs
            if ev is not None:
                ev[2].record(st if st is not None else torch.cuda.current_stream())
                events.append(ev)
        return cur, limbs
