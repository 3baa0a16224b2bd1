"""Helpers shared by the GPU tests (not collected as tests)."""
import numpy as np


def torch():
    import torch as t
    return t


def seeds_tensor(seeds):
    t = torch()
    return t.from_numpy(np.asarray(seeds, dtype=np.uint64).view(np.int64)).cuda()


def rel_err(got, ref):
    """Normwise relative error max|got - ref| / max|ref| (per last axis)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    num = np.abs(got - ref).max(axis=-1)
    den = np.maximum(np.abs(ref).max(axis=-1), 1e-30)
    return num / den


def bf16_to_f64(t):
    """torch bf16 tensor -> float64 numpy (exact)."""
    return t.float().cpu().numpy().astype(np.float64)


def sample_gpu(rgd, z_np, T, pmin, seeds, ctr=0, stream0=0, draws=1):
    t = torch()
    z = t.from_numpy(np.ascontiguousarray(z_np, dtype=np.float32)).cuda()
    R, V = z.shape
    ws = t.empty(rgd.sampler_workspace_bytes(R, V), dtype=t.uint8, device="cuda")
    out = t.full((R, draws), -1, dtype=t.int32, device="cuda")
    rgd.kernel_sample(z, T, pmin, seeds_tensor(seeds), ctr, stream0, draws, ws, out)
    t.cuda.synchronize()
    return out.cpu().numpy()


def argmax_gpu(rgd, z_np):
    t = torch()
    z = t.from_numpy(np.ascontiguousarray(z_np, dtype=np.float32)).cuda()
    R, V = z.shape
    ws = t.empty(rgd.sampler_workspace_bytes(R, V), dtype=t.uint8, device="cuda")
    out = t.full((R,), -1, dtype=t.int32, device="cuda")
    rgd.kernel_argmax(z, ws, out)
    t.cuda.synchronize()
    return out.cpu().numpy()


MARGIN = 1e-4

# judged draws per test case: {case: {"exact", "margin-equal", "margin-diff", "draws"}},
# written to gpurun_out/margin_cases.json at the end of a session that judged any
MARGIN_REPORT = {}


class Tally:
    """Verdict counts of the draws judged under one name.  close() records them
    in MARGIN_REPORT, prints them and bounds the margin-diff draws (tokens that
    differ from the oracle's in a margin case) to max(1, frac * draws)."""

    def __init__(self, name):
        self.name = name
        self.c = {"exact": 0, "margin-equal": 0, "margin-diff": 0}

    def add(self, verdict):
        self.c[verdict] += 1
        return verdict

    def close(self, max_diff_frac=0.01):
        n = sum(self.c.values())
        MARGIN_REPORT[self.name] = dict(self.c, draws=n)
        print(self.name, self.c)
        assert self.c["margin-diff"] <= max(1, int(max_diff_frac * n)), (self.name, self.c)
        return self.c


def _robust(w, kept, amb, u, tok, margin):
    """True when the oracle's draw `tok` cannot change under any flip of the
    mask decisions within the margin (tokens in `amb`) or a relative error of
    `margin` in the running sums: tok itself is not ambiguous and u * W lies
    inside tok's CDF interval by more than twice the ambiguous weight plus
    margin * W on both sides.  Such draws must match exactly even though some
    mask decision elsewhere is a near tie."""
    if amb[tok]:
        return False
    wk = np.where(kept, w, 0.0)
    W = wk.sum()
    lo = wk[:tok].sum()
    hi = lo + wk[tok]
    t = u * W
    slack = 2.0 * w[amb].sum() + margin * W
    return t - lo > slack and hi - t > slack


def judge_draw(z, T, pmin, u, got, margin=MARGIN):
    """Classifies one GPU draw against the oracle on the same logits.

    Outside margin cases (oracle CDF margin and min-p logit margin >= margin)
    the token must be identical.  In a margin case the GPU token must still be
    a valid outcome: kept under the mask relaxed by the margin, with its CDF
    interval within margin * W (plus the weight of tokens whose mask decision
    is itself within the margin) of u * W.
    Returns "exact", "margin-equal" or "margin-diff"."""
    from oracle import sampler
    d = sampler.sample_minp(z, T, pmin, u)
    w, _ = sampler.minp_weights(z, T, pmin)
    lw = np.log(np.maximum(w, 1e-300))
    amb = np.abs(lw - np.log(pmin)) < margin if pmin > 0 else np.zeros_like(w, bool)
    if (d.cdf_margin >= margin and d.logit_margin >= margin) or _robust(w, w >= pmin, amb, u, d.token, margin):
        assert got == d.token, (got, d)
        return "exact"
    if got == d.token:
        return "margin-equal"
    kept = w >= pmin * np.exp(-margin)
    assert kept[got], ("token outside the relaxed min-p set", got)
    wk = np.where(w >= pmin, w, 0.0)
    W = wk.sum()
    c = np.cumsum(wk)
    lo, hi = c[got] - wk[got], c[got]
    t = u * W
    slack = margin * W + w[amb].sum()
    assert lo - slack <= t <= hi + slack, ("draw too far from u*W", got, d.token)
    return "margin-diff"


def judge_draw_pless(z, T, u, got, margin=MARGIN):
    """judge_draw for the p-less rule (keep p_i >= sum_j p_j^2): identical token
    outside margin cases (CDF margin and |ln p_i - ln sum p^2| >= margin for
    every token), otherwise a valid outcome under the mask relaxed by the
    margin."""
    from oracle import pless
    d = pless.sample_pless(z, T, u)
    p, thr, _ = pless.pless_probabilities(z, T)
    lp = np.log(np.maximum(p, 1e-300))
    amb = np.abs(lp - np.log(thr)) < margin
    if (d.cdf_margin >= margin and d.logit_margin >= margin) or _robust(p, p >= thr, amb, u, d.token, margin):
        assert got == d.token, (got, d)
        return "exact"
    if got == d.token:
        return "margin-equal"
    assert p[got] >= thr * np.exp(-margin), ("token outside the relaxed p-less set", got)
    pk = np.where(p >= thr, p, 0.0)
    W = pk.sum()
    c = np.cumsum(pk)
    lo, hi = c[got] - pk[got], c[got]
    t = u * W
    slack = margin * W + p[amb].sum()
    assert lo - slack <= t <= hi + slack, ("draw too far from u*W", got, d.token)
    return "margin-diff"
