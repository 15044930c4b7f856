"""Comparison rules between the HIP path and the oracle, and host<->device
plumbing for the GPU tests.

Tolerances:
  * refresh, int8 codes, fp32 scales, gathered bf16: bit for bit (one correct
    result exists for identical inputs);
  * Adam fp32 master / moments (see assert_adam_close): the relative error of
    element i is |a - r| / max(|r|, tau) and must stay within 1e-5, with
    tau = lr for the master weights (one update's size) and
    tau = 1e-6 * max|r| for the moments (the strict rule).  The first
    moment is a sum of two terms of either sign; where they cancel, the
    strict rule asks for more relative precision than a binary32 sum can keep,
    so an element that misses it passes only within the sum's own forward
    error bound, 4 * 2^-24 times the size of the terms summed since the common
    state (derived in first_moment_bound);
  * Adam bf16 primary: the exact rounding of the kernel's own fp32 master,
    and within 1 bf16 ulp of the oracle's; an element of the oracle below lr
    in magnitude that is further apart is accepted only when the masters
    themselves pass their rule, so the difference is the masters' own.
Every comparison counts, per array, the elements equal bit for bit, those
passing the strict rule, and those passing only the derived bound; over a
whole partition the number passing only the bound is capped (RELAXED_CAP).
"""
import threading

import numpy as np
import torch

import oracle

REL_TOL = 1e-5
U32 = 2.0 ** -24  # unit roundoff of binary32 round-to-nearest
# First moment: kernel and oracle may differ by at most FIRST_MOMENT_K * U32
# times the size of the terms summed (plus FIRST_MOMENT_ABS for results in
# the subnormal range); derived in first_moment_bound.
FIRST_MOMENT_K = 4.0 * (1.0 + 2.0 ** -16)
FIRST_MOMENT_ABS = 2.0 ** -148
# At most this fraction of an array's elements may pass only the derived
# bound (the first moment: where its two terms cancel; the bf16 primary: an
# oracle value below lr whose rounding differs by more than 1 ulp).
RELAXED_CAP = {"master": 0.0, "exp_avg": 1e-2, "exp_avg_sq": 0.0, "bf16": 2e-6}

# Every comparison's counts, in call order: (label, {array: counts}).
ADAM_COUNTS = []
_COUNTS_LOCK = threading.Lock()


def rel_err(a, r, tau):
    a = np.asarray(a, np.float64)
    r = np.asarray(r, np.float64)
    with np.errstate(invalid="ignore", divide="ignore"):
        e = np.abs(a - r) / np.maximum(np.abs(r), tau)
    return np.where(a == r, 0.0, e)  # equal infinities are no error


def assert_same_nan(a, r, what):
    na, nr = np.isnan(a), np.isnan(r)
    assert np.array_equal(na, nr), "%s: NaN positions differ (%d vs %d)" % (what, na.sum(), nr.sum())
    return ~na


def first_moment_scale(prev, g, hp, adamw=True):
    """beta1*|m| + (1-beta1)*|g'| of one step (g' = g + wd*p in the L2 form):
    the size of the two terms the first-moment update sums."""
    b1 = float(hp["beta1"])
    gabs = np.abs(np.asarray(g, np.float64))
    if not adamw:
        gabs = gabs + float(hp["weight_decay"]) * np.abs(np.asarray(prev[0], np.float64))
    return b1 * np.abs(np.asarray(prev[1], np.float64)) + (1.0 - b1) * gabs


def first_moment_bound(scale):
    """Largest |kernel - oracle| of the first moment, given the size S of
    the terms summed (first_moment_scale, or MomentTolerance over several
    steps).  Forward error of one step: the kernel forms
    m' = fma(b1, m, RN(c * g')) with g' = g (AdamW) or RN(g + wd*p) (L2,
    one fma), the oracle the exact sum rounded once to binary32.  The
    operand roundings differ from the exact terms by at most 2 U c|g'|, and
    each side's final rounding adds at most U |m'| <= U S, so one step adds
    at most 4 U S; an error carried in m from earlier steps is multiplied by
    b1 < 1, which is how MomentTolerance discounts S.  The factor
    (1 + 2^-16) covers the second-order terms (the roundings of the
    rounded terms, the oracle's binary64 sum), and a subnormal result
    adds at most 2^-148 absolute."""
    return FIRST_MOMENT_K * U32 * np.asarray(scale, np.float64) + FIRST_MOMENT_ABS


class MomentTolerance:
    """Running size of the first moment's terms over several steps taken
    from a common starting state: an error made at step k decays by beta1
    per later step, so the size is the beta1-discounted sum of the per-step
    term sizes, S_t = beta1 * S_(t-1) + first_moment_scale_t.

    In the L2 form the gradient that enters the moment is g + wd*p, so a
    difference d between the two sides' master weights before a step enters
    the first moment as (1 - beta1) * wd * |d| beyond the roundings;
    step(p_diff=d) adds that term, expressed in the units of S
    (first_moment_bound multiplies S by FIRST_MOMENT_K * U32)."""

    def __init__(self):
        self.s = None

    def step(self, prev, g, hp, adamw=True, p_diff=None):
        cur = first_moment_scale(prev, g, hp, adamw)
        if p_diff is not None and not adamw:
            carried = ((1.0 - float(hp["beta1"])) * float(hp["weight_decay"])
                       * np.abs(np.asarray(p_diff, np.float64)))
            cur = cur + carried * (1.0 + U32) / (FIRST_MOMENT_K * U32)
        self.s = cur if self.s is None else float(hp["beta1"]) * self.s + cur
        return self.s


def _counts(n, bitwise, strict, relaxed, fail):
    return dict(n=int(n), bitwise=int(bitwise), strict=int(strict), relaxed_only=int(relaxed),
                fail=int(fail))


def adam_counts(got, ref, lr, prev=None, g=None, hp=None, adamw=True, m_tau=None):
    """Per array of (master, exp_avg, exp_avg_sq, bf16): the number of
    elements compared, equal bit for bit, passing the strict rule, passing
    only the derived bound, and failing both.  NaN positions must agree
    (checked by assert_adam_close); NaN elements count as equal."""
    gp, gm, gv, gb = (np.asarray(x) for x in got)
    rp, rm, rv, rb = (np.asarray(x) for x in ref)
    out = {}
    tiny = np.finfo(np.float32).tiny
    # master weights: tau = lr, no relaxation
    ok = ~np.isnan(rp)
    bit = np.sum(gp.view(np.uint32) == rp.view(np.uint32)) + np.sum(~ok & np.isnan(gp))
    strict = rel_err(gp[ok], rp[ok], lr) <= REL_TOL
    out["master"] = _counts(gp.size, bit, strict.sum() + (~ok).sum(), 0, (~strict).sum())
    master_ok = np.ones(gp.size, bool)
    master_ok[ok] = strict
    # moments: tau = 1e-6 max|r|; the first moment may fall back on the
    # forward error bound of its sum
    if m_tau is None and prev is not None:
        m_tau = first_moment_scale(prev, g, hp, adamw)
    for a, r, name in ((gm, rm, "exp_avg"), (gv, rv, "exp_avg_sq")):
        ok = ~np.isnan(r)
        bit = np.sum(a.view(np.uint32) == r.view(np.uint32)) + np.sum(~ok & np.isnan(a))
        if not ok.any():
            out[name] = _counts(a.size, bit, a.size, 0, 0)
            continue
        tau = max(1e-6 * float(np.abs(r[ok]).max()), tiny)
        strict = rel_err(a[ok], r[ok], tau) <= REL_TOL
        relaxed = np.zeros_like(strict)
        if name == "exp_avg" and m_tau is not None:
            with np.errstate(invalid="ignore"):  # equal infinities
                diff = np.abs(a[ok].astype(np.float64) - r[ok].astype(np.float64))
            bound = first_moment_bound(np.broadcast_to(np.asarray(m_tau), a.shape)[ok])
            relaxed = ~strict & (diff <= bound)
        out[name] = _counts(a.size, bit, strict.sum() + (~ok).sum(), relaxed.sum(),
                            (~strict & ~relaxed).sum())
    # bf16 primary: within 1 ulp of the oracle's; below lr, further apart
    # only where the masters passed their rule
    fin = np.isfinite(rp) & np.isfinite(gp)
    d = np.abs(bf16_ordered(gb) - bf16_ordered(rb))
    strict = ~fin | (d <= 1)
    relaxed = ~strict & (np.abs(rp) < lr) & master_ok
    out["bf16"] = _counts(gb.size, np.sum(gb == rb), strict.sum(), relaxed.sum(),
                          (~strict & ~relaxed).sum())
    return out


def assert_adam_close(got, ref, lr, what="", prev=None, g=None, hp=None, adamw=True,
                      m_tau=None, cap=False, record=False):
    """got/ref: (p, m, v, bf16) tuples of numpy arrays after the same steps
    from a common state.

    Master weights: relative error within 1e-5 with tau = lr.  First moment:
    within 1e-5 with tau = 1e-6 max|m|, or else within first_moment_bound of
    the terms' size, taken from m_tau if given (see MomentTolerance), else
    from the step's inputs when given (prev = (p, m, v) before the step,
    gradient g, hyperparameters); without either (a zero first moment before
    the step: m = (1-beta1)*g involves no sum) only the strict rule applies.
    Second moment (a sum of non-negative terms): tau = 1e-6 max|v|.  bf16
    primary: see assert_bf16_primary.  Returns the counts of adam_counts;
    with cap=True the elements passing only the derived bound are capped
    (assert_relaxed_capped), with record=True the counts are also kept in
    ADAM_COUNTS under `what`."""
    gp, gm, gv, gb = got
    rp, rm, rv, rb = ref
    for a, r, name in ((gp, rp, "master"), (gm, rm, "exp_avg"), (gv, rv, "exp_avg_sq")):
        assert_same_nan(a, r, what + " " + name)
    assert_bf16_primary(gb, gp, rb, rp, what + " bf16")
    c = adam_counts(got, ref, lr, prev, g, hp, adamw, m_tau)
    for name, k in c.items():
        assert k["fail"] == 0, "%s %s: %d of %d elements out of bound%s" % (
            what, name, k["fail"], k["n"], _worst(got, ref, lr, name, m_tau))
    if cap:
        assert_relaxed_capped(c, what)
    if record:
        with _COUNTS_LOCK:
            ADAM_COUNTS.append((what, c))
    return c


def assert_relaxed_capped(c, what):
    """At most RELAXED_CAP[array] * n elements pass only the derived bound."""
    for name, k in c.items():
        cap = int(RELAXED_CAP[name] * k["n"])
        assert k["relaxed_only"] <= cap, "%s %s: %d of %d elements pass only the derived " \
            "bound (cap %d)" % (what, name, k["relaxed_only"], k["n"], cap)


def _worst(got, ref, lr, name, m_tau):
    i = {"master": 0, "exp_avg": 1, "exp_avg_sq": 2, "bf16": 3}[name]
    a, r = np.asarray(got[i]), np.asarray(ref[i])
    if name == "bf16":
        d = np.abs(bf16_ordered(a) - bf16_ordered(r))
        k = int(np.argmax(d))
        return "; worst at %d: %d ulp (%#x vs %#x)" % (k, d[k], int(a[k]), int(r[k]))
    diff = np.abs(a.astype(np.float64) - r.astype(np.float64))
    diff[np.isnan(diff)] = 0.0
    k = int(np.argmax(diff / np.maximum(np.abs(r.astype(np.float64)), lr if i == 0 else 1e-30)))
    return "; worst at %d: got %r want %r" % (k, float(a[k]), float(r[k]))


def merge_counts(parts):
    """Sum per-array counts of several comparisons (chunks of one array)."""
    out = {}
    for c in parts:
        for name, k in c.items():
            acc = out.setdefault(name, dict.fromkeys(k, 0))
            for key, val in k.items():
                acc[key] += val
    return out


class ChunkedAdam:
    """The oracle's Adam state for a whole partition, kept in chunks that a
    pool of host threads steps and checks side by side (the oracle's calls
    and numpy's array work release the GIL).  Each chunk carries its own
    first-moment tolerance (MomentTolerance) from the common start."""

    def __init__(self, p0, hp, ex, parts=64):
        n = p0.size
        step = -(-n // parts)
        self.rs = [(a, min(n, a + step)) for a in range(0, n, step)]
        self.hp, self.ex, self.t = hp, ex, 0
        self.st = [dict(p=p0[a:b].copy(), m=np.zeros(b - a, np.float32),
                        v=np.zeros(b - a, np.float32), mt=MomentTolerance())
                   for a, b in self.rs]

    def step(self, g):
        self.t += 1

        def one(k):
            st, (a, b) = self.st[k], self.rs[k]
            st["tau"] = st["mt"].step((st["p"], st["m"], st["v"]), g[a:b], self.hp)
            st["p"], st["m"], st["v"], st["b"] = oracle.adam_step(
                st["p"], st["m"], st["v"], g[a:b], step=self.t, **self.hp)

        list(self.ex.map(one, range(len(self.rs))))

    def check(self, got, what):
        """got: whole (p, m, v, bf16) arrays, `self.t` steps after the start.
        Returns the counts over the whole partition, capped
        (assert_relaxed_capped) and recorded in ADAM_COUNTS."""
        def one(k):
            st, (a, b) = self.st[k], self.rs[k]
            return assert_adam_close(tuple(x[a:b] for x in got),
                                     (st["p"], st["m"], st["v"], st["b"]), self.hp["lr"],
                                     "%s [%d, %d)" % (what, a, b), m_tau=st["tau"])

        c = merge_counts(self.ex.map(one, range(len(self.rs))))
        assert_relaxed_capped(c, what)
        with _COUNTS_LOCK:
            ADAM_COUNTS.append((what, c))
        return c


def bf16_value(h):
    return (np.asarray(h, np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def assert_bf16_primary(gb, gp, rb, rp, what):
    """The emitted bf16 primary is exactly the round-to-nearest-even of the
    kernel's own fp32 master (torch's CPU conversion as the reference
    rounding, NaN canonical), with NaN where the oracle has NaN.  Its
    distance to the oracle's bf16 is counted by adam_counts."""
    isn = np.isnan(gp)
    lib = torch.from_numpy(np.ascontiguousarray(gp)).to(torch.bfloat16).view(torch.int16)
    lib = lib.numpy().view(np.uint16)
    assert_bits_equal(gb[~isn], lib[~isn], what + " vs rounding of the kernel's master")
    assert np.all(gb[isn] == 0x7FC0), what + ": NaN not canonical"
    rn = np.isnan(rp)
    assert np.array_equal(isn, rn), what + ": NaN positions differ"
    assert np.all(np.asarray(rb)[rn] == 0x7FC0), what + ": oracle NaN not canonical"


def bf16_ordered(h):
    h = np.asarray(h, np.uint16).astype(np.int32)
    mag = h & 0x7FFF
    return np.where(h & 0x8000, -mag, mag)


def bf16_is_nan(h):
    h = np.asarray(h, np.uint16)
    return ((h & 0x7F80) == 0x7F80) & ((h & 0x007F) != 0)


def assert_bf16_within_ulp(got, ref, what=""):
    gn, rn = bf16_is_nan(got), bf16_is_nan(ref)
    assert np.array_equal(gn, rn), what + ": NaN positions differ"
    assert np.all(np.asarray(got)[gn] == 0x7FC0), what + ": NaN not canonical"
    d = np.abs(bf16_ordered(got)[~gn] - bf16_ordered(ref)[~gn])
    assert d.size == 0 or d.max() <= 1, "%s: bf16 differs by %d ulp" % (what, d.max())


def assert_bits_equal(got, ref, what=""):
    got = np.asarray(got)
    ref = np.asarray(ref)
    assert got.shape == ref.shape, "%s: shape %s vs %s" % (what, got.shape, ref.shape)
    g = got.view(np.uint8) if got.dtype.itemsize else got
    r = ref.view(np.uint8) if ref.dtype.itemsize else ref
    if not np.array_equal(g, r):
        gw = got.view({1: np.uint8, 2: np.uint16, 4: np.uint32}[got.dtype.itemsize])
        rw = ref.view({1: np.uint8, 2: np.uint16, 4: np.uint32}[ref.dtype.itemsize])
        bad = np.nonzero(gw != rw)[0]
        raise AssertionError("%s: %d of %d elements differ; first at %d: got %#x want %#x"
                             % (what, bad.size, got.size, bad[0], int(gw[bad[0]]),
                                int(rw[bad[0]])))


# ---------------------------------------------------------------------------
# host <-> device
# ---------------------------------------------------------------------------
_TORCH_OF = {np.dtype(np.float32): torch.float32, np.dtype(np.int8): torch.int8,
             np.dtype(np.uint16): torch.int16}


def to_dev(a, device="cuda", pad=0):
    """numpy -> new contiguous device tensor (uint16 travels as int16);
    ``pad`` extra zero elements are allocated in front, and the returned
    tensor is the view that starts ``pad`` elements in (misaligned views)."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    t = torch.from_numpy(a)
    if pad:
        buf = torch.zeros(a.size + pad, dtype=t.dtype, device=device)
        buf[pad:].copy_(t.to(device))
        return buf[pad:]
    return t.to(device).contiguous()


def empty_dev(n, np_dtype, device="cuda", pad=0, fill=None):
    dt = _TORCH_OF[np.dtype(np_dtype)]
    buf = torch.empty(n + pad, dtype=dt, device=device)
    if fill is not None:
        buf.fill_(fill)
    return buf[pad:] if pad else buf


def to_host(t, np_dtype):
    a = t.detach().cpu().numpy()
    return a.view(np_dtype)
