"""Helpers shared by the GPU tests: host/device conversions and ulp distances."""
import numpy as np


def torch():
    import torch as _t

    return _t


def to_dev_bf16(bits: np.ndarray):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16)).view(t.bfloat16).cuda()


def to_dev(a: np.ndarray):
    t = torch()
    if a.dtype == np.uint16:
        return to_dev_bf16(a)
    return t.from_numpy(np.ascontiguousarray(a)).cuda()


def to_host(x) -> np.ndarray:
    t = torch()
    if x.dtype == t.bfloat16:
        return x.view(t.int16).cpu().numpy().view(np.uint16)
    return x.cpu().numpy()


def _ordered32(a: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.int64)
    neg = u >= 0x80000000
    return np.where(neg, 0x80000000 - u, u)        # -0 and +0 both map to 0


def ulp_f32(a, b) -> np.ndarray:
    """Distance in fp32 ulps (units in the last place) between finite arrays."""
    return np.abs(_ordered32(a) - _ordered32(b))


def ulp_bf16(a_bits, b_bits) -> np.ndarray:
    u = np.ascontiguousarray(a_bits, dtype=np.uint16).astype(np.int64)
    v = np.ascontiguousarray(b_bits, dtype=np.uint16).astype(np.int64)
    ou = np.where(u >= 0x8000, 0x8000 - u, u)
    ov = np.where(v >= 0x8000, 0x8000 - v, v)
    return np.abs(ou - ov)


def normals_within_2ulp(got: np.ndarray, ref: np.ndarray) -> bool:
    """|got - ref| <= 2 ulp32(ref), with ulp32(0) = 2^-149 (zeros must be exact)."""
    got = got.astype(np.float64)
    ref32 = ref.astype(np.float32)
    ulp = np.where(ref32 == 0, 2.0 ** -149, np.spacing(np.abs(ref32)).astype(np.float64))
    return bool(np.all(np.abs(got - ref.astype(np.float64)) <= 2 * ulp))


def f32_close(got, ref, rtol=1e-5, atol=1e-7) -> bool:
    """|got - ref| <= rtol |ref| + atol elementwise."""
    g = got.astype(np.float64)
    r = ref.astype(np.float64)
    return bool(np.all(np.abs(g - r) <= rtol * np.abs(r) + atol))


def bf16_value(bits) -> np.ndarray:
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def bf16_ulp(x: np.ndarray) -> np.ndarray:
    """Spacing of bf16 numbers at |x| (8 significand bits)."""
    ax = np.abs(x.astype(np.float64))
    _, e = np.frexp(np.where(ax == 0, 2.0 ** -126, ax))
    return np.ldexp(1.0, e - 8)


def bf16_close(got_bits, ref_bits) -> bool:
    """|got - ref| <= 1 bf16 ulp(ref): the bar for perturbed bf16 weights (one
    fp32 fma, then the rounding to bf16, on both sides)."""
    g = bf16_value(got_bits).astype(np.float64)
    r = bf16_value(ref_bits).astype(np.float64)
    return bool(np.all(np.abs(g - r) <= bf16_ulp(r)))


def update_slack(orc, seeds, signs, rnorm, step, j) -> np.ndarray:
    """(n_streams + 2) 2^-24 |step| sum_u |c_u z_u(j)| at noise positions j:
    how far the device's fp32 accumulation of an update (Eq. 13) can drift
    from the oracle's fp64 one.  The device rounds each coefficient
    c_u = sum of sign * rnorm over the members of stream u, and the step, to
    fp32 (2^-24 relative each) and adds the n_streams products c_u z_u with
    fused multiply-adds, each rounding the running sum once (at most
    2^-24 sum_u |c_u z_u| each)."""
    coef = {}
    for sd, sg, r in zip(seeds, signs, rnorm):
        coef[int(sd)] = coef.get(int(sd), 0.0) + float(sg) * float(r)
    j = np.asarray(j, dtype=np.int64)
    tot = np.zeros(len(j))
    for sd, c in coef.items():
        z = np.array([orc.normal(sd, int(x)) for x in j], dtype=np.float64)
        tot += abs(c) * np.abs(z)
    return (len(coef) + 2) * 2.0 ** -24 * abs(float(step)) * tot


def update_step_size(alpha, sigma, n, scale_mode) -> float:
    """alpha / (n sigma) (scale mode 0) or alpha / n (scale mode 1)."""
    return float(alpha) / (n * float(sigma)) if scale_mode == 0 else float(alpha) / n


def bf16_update_close(got_bits, ref_bits, slack_at) -> bool:
    """The bar for bf16 weights after an update, per element k:
        |got - ref| <= ulp_bf16(max(|got|, |ref|)) + 2^-23 |ref| + slack_at(k).
    The first term is the two roundings to bf16, the second the two fp32
    roundings before them, and slack_at(k) (update_slack at element k's noise
    position) the fp32 accumulation.  slack_at is only evaluated at the
    elements the first two terms do not cover."""
    g = bf16_value(got_bits).astype(np.float64)
    r = bf16_value(ref_bits).astype(np.float64)
    base = bf16_ulp(np.maximum(np.abs(g), np.abs(r))) + 2.0 ** -23 * np.abs(r)
    over = np.nonzero(np.abs(g - r) > base)[0]
    if over.size == 0:
        return True
    return bool(np.all(np.abs(g[over] - r[over]) <= base[over] + slack_at(over)))


def describe_mismatch(got, ref) -> str:
    g = got.astype(np.float64)
    r = ref.astype(np.float64)
    k = int(np.argmax(np.abs(g - r)))
    return f"max |diff| {abs(g[k] - r[k]):.3e} at {k}: got {g[k]!r} ref {r[k]!r}"


def zscore_close(got, ref, r, group=None) -> bool:
    """Z-scores of the device against the oracle's, per element:
        |got - ref| <= ulp32(ref) + 2 (c + 8) 2^-53 ((1 + |z|) A / s + |z|),
    with c the size, A the mean |r| and s the population standard deviation of
    the element's group (fp64), z = ref.  The oracle sums each group
    sequentially, the device in another fixed order (64 lane-strided partial
    sums and a butterfly); each fp64 sum of c terms is within (c - 1) 2^-53 A c
    of the exact one, so the means differ by at most about 2 (c + 8) 2^-53 A
    and the deviations' relative error is about as large.  Carried through
    (r - mu) / s that bounds the fp64 quotients' difference, and the rounding
    to fp32 adds at most one ulp.  A group with s = 0 must give exact zeros."""
    got = np.asarray(got, dtype=np.float64)
    ref32 = np.asarray(ref, dtype=np.float32)
    ref = ref32.astype(np.float64)
    r = np.asarray(r, dtype=np.float64)
    g = np.zeros(len(r), dtype=np.int64) if group is None else np.asarray(group)
    bound = np.zeros(len(r))
    for k in np.unique(g):
        m = g == k
        c = int(m.sum())
        mu = r[m].mean()
        s = np.sqrt(((r[m] - mu) ** 2).mean())
        if s == 0:
            continue                                     # outputs must be exactly 0
        z = np.abs(ref[m])
        bound[m] = 2 * (c + 8) * 2.0 ** -53 * ((1 + z) * np.abs(r[m]).mean() / s + z)
    ulp = np.where(ref32 == 0, 2.0 ** -149, np.spacing(np.abs(ref32)).astype(np.float64))
    ok = np.abs(got - ref) <= np.where(bound > 0, ulp + bound, 0.0)
    return bool(np.all(ok))
