"""Comparison rules between the HIP path and the oracle, and host<->device
plumbing for the GPU tests.

Tolerances:
  * refresh, int8 codes, fp32 scales, gathered bf16: bit for bit (one correct
    result exists for identical inputs);
  * Adam fp32 master / moments: max relative error 1e-5, with the relative
    error of element i taken as |a - r| / max(|r|, tau): tau = lr per step
    since the common state for the master weights (a weight that lands within
    the updates' reach of zero has no meaningful relative error); for the
    first moment tau is the size of the terms its updates summed, discounted
    by beta1 per step (see assert_adam_close, MomentTolerance); for the second
    moment (a sum of non-negative terms) tau = 1e-6 * max|v| only guards
    exact zeros;
  * Adam bf16 primary: the exact rounding of the kernel's own fp32 master,
    and within 1 bf16 ulp of the oracle's (the fp32 results may differ in the
    last bits, which can move a value across a bf16 rounding boundary) where
    the master's relative criterion applies; see assert_bf16_primary.
"""
import numpy as np
import torch

import oracle

REL_TOL = 1e-5


def rel_err(a, r, tau):
    a = np.asarray(a, np.float64)
    r = np.asarray(r, np.float64)
    with np.errstate(invalid="ignore"):
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


class MomentTolerance:
    """Running tolerance of the first moment over several steps taken from a
    common starting state: an error made at step k decays by beta1 per later
    step, so the tolerance is the beta1-discounted sum of the per-step term
    sizes, S_t = beta1 * S_(t-1) + first_moment_scale_t."""

    def __init__(self):
        self.s = None

    def step(self, prev, g, hp, adamw=True):
        cur = first_moment_scale(prev, g, hp, adamw)
        self.s = cur if self.s is None else float(hp["beta1"]) * self.s + cur
        return self.s


def assert_adam_close(got, ref, lr, what="", prev=None, g=None, hp=None, adamw=True, steps=1,
                      m_tau=None):
    """got/ref: (p, m, v, bf16) tuples of numpy arrays, `steps` steps after
    the kernel and the oracle last shared their state.

    Master weights: tau = steps * lr (a weight within the distance the
    updates can move it of zero carries no meaningful relative error, and the
    rounding of every step since the common state adds to the absolute one).
    First moment: tau = m_tau if given (see MomentTolerance), else, when the
    step's inputs are given (prev = (p, m, v) before the step, gradient g,
    hyperparameters), the size of the two terms it sums; without them (zero
    first moment before the step: m = (1-beta1)*g involves no sum)
    tau = 1e-6 * max|m| guards values at zero.  Second moment (a sum of
    non-negative terms): tau = 1e-6 * max|v|."""
    gp, gm, gv, gb = got
    rp, rm, rv, rb = ref
    tau_p = lr * steps
    ok = assert_same_nan(gp, rp, what + " master")
    e = rel_err(gp[ok], rp[ok], tau_p)
    assert e.size == 0 or e.max() <= REL_TOL, "%s master rel err %.3g" % (what, e.max())
    tiny = np.finfo(np.float32).tiny
    if m_tau is None and prev is not None:
        m_tau = first_moment_scale(prev, g, hp, adamw)
    for a, r, name in ((gm, rm, "exp_avg"), (gv, rv, "exp_avg_sq")):
        ok = assert_same_nan(a, r, what + " " + name)
        if not ok.any():
            continue
        if name == "exp_avg" and m_tau is not None:
            tau = np.maximum(np.asarray(m_tau)[ok], tiny)
        else:
            tau = max(1e-6 * float(np.abs(r[ok]).max()), tiny)
        e = rel_err(a[ok], r[ok], tau)
        assert e.max() <= REL_TOL, "%s %s rel err %.3g" % (what, name, e.max())
    assert_bf16_primary(gb, gp, rb, rp, tau_p, what + " bf16")


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
        """got: whole (p, m, v, bf16) arrays, `self.t` steps after the start."""
        def one(k):
            st, (a, b) = self.st[k], self.rs[k]
            assert_adam_close(tuple(x[a:b] for x in got), (st["p"], st["m"], st["v"], st["b"]),
                              self.hp["lr"], "%s [%d, %d)" % (what, a, b), steps=self.t,
                              m_tau=st["tau"])

        list(self.ex.map(one, range(len(self.rs))))


def bf16_value(h):
    return (np.asarray(h, np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def assert_bf16_primary(gb, gp, rb, rp, tau, what):
    """The emitted bf16 primary is (a) exactly the round-to-nearest-even of the
    kernel's own fp32 master (torch's CPU conversion as the reference
    rounding, NaN canonical), and (b) within 1 bf16 ulp of the oracle's where
    the master's relative criterion applies (|r| >= tau); nearer zero, where
    the masters may differ by up to 1e-5 * tau, the two bf16 values differ by
    no more than that plus half an ulp of each."""
    isn = np.isnan(gp)
    lib = torch.from_numpy(np.ascontiguousarray(gp)).to(torch.bfloat16).view(torch.int16)
    lib = lib.numpy().view(np.uint16)
    assert_bits_equal(gb[~isn], lib[~isn], what + " vs rounding of the kernel's master")
    assert np.all(gb[isn] == 0x7FC0), what + ": NaN not canonical"
    rn = np.isnan(rp)
    assert np.array_equal(isn, rn), what + ": NaN positions differ"
    fin = ~rn & np.isfinite(rp)
    well = fin & (np.abs(rp) >= tau)
    assert_bf16_within_ulp(gb[well], rb[well], what)
    near = fin & ~well
    if near.any():
        gv = bf16_value(gb[near]).astype(np.float64)
        rv = bf16_value(rb[near]).astype(np.float64)
        half = lambda x: np.spacing(np.abs(x).astype(np.float32)).astype(np.float64) * 32768.0
        tol = REL_TOL * tau + half(gv) + half(rv)
        assert np.all(np.abs(gv - rv) <= tol), what + ": bf16 near zero out of bound"


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
