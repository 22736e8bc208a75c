"""Element-wise checks of one forward stage fed identical inputs on both sides (test infrastructure).

Each stage of a layer (RMSNorm, QKV + RoPE, attention, residual projections, SwiGLU) is evaluated
by the oracle's stage function on the GPU's own stage inputs, so the only difference left is the
GPU's float32 arithmetic. For every output element an a-priori bound E on that float32 error is
derived from the operation's length and operand magnitudes (standard floating-point error
analysis: a sum of n terms evaluated in any order with each addition rounded has error at most
gamma_n * sum |terms|, gamma_n = n u / (1 - n u)):

* float32 outputs (the residual stream): |gpu - exact| <= E;
* bf16 outputs: the GPU's value is the bf16 rounding of some float32 value within E of the exact
  one, i.e. it lies in [bf16(exact - E), bf16(exact + E)]; it is never more than one bf16 ulp
  from bf16(exact) unless E itself exceeds half an ulp (values near zero after cancellation);
  elements where it differs from bf16(exact) (a rounding flip, only possible where the exact value
  lies within E of a rounding midpoint) are counted and their fraction is bounded.

Unit roundoffs: U = 2^-24 for elementwise float32 operations; U_ACC = 2^-23 for MFMA and reduction
accumulations (twice the round-to-nearest unit, so the bound also holds if an accumulation step
truncates).
"""
import numpy as np

from oracle.numerics import bf16_round

U = 2.0 ** -24
U_ACC = 2.0 ** -23
MAX_FLIP_FRACTION = 0.02   # bf16 outputs: at most this fraction of elements may round the other way


def gamma(n, u=U_ACC):
    return n * u / (1.0 - n * u)


def bf16_bits_to_f64(bits):
    b = np.asarray(bits).view(np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def _ordered(bits):
    """bf16 bit patterns -> integers in the order of their values (+0 and -0 both 0)."""
    b = np.asarray(bits).view(np.uint16).astype(np.int64)
    mag = b & 0x7FFF
    return np.where(b & 0x8000, -mag, mag)


def _bits_of(x):
    """bf16 bit patterns of float64 values that are exactly representable in bf16."""
    return (np.asarray(x, np.float64).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)


def check_bf16(name, gpu_bits, exact, E, report, max_flip=MAX_FLIP_FRACTION):
    """GPU bf16 output vs the exact stage value with per-element float32 error bound E."""
    exact = np.asarray(exact, np.float64)
    E = np.broadcast_to(np.asarray(E, np.float64), exact.shape)
    g = bf16_bits_to_f64(gpu_bits).reshape(exact.shape)
    nearest = bf16_round(exact)
    lo, hi = bf16_round(exact - E), bf16_round(exact + E)
    inside = (g >= lo) & (g <= hi)
    ulps = np.abs(_ordered(np.asarray(gpu_bits).reshape(exact.shape)) - _ordered(_bits_of(nearest)))
    flips = g != nearest
    frac = float(flips.mean()) if flips.size else 0.0
    report[name] = {"elements": int(flips.size), "flips": int(flips.sum()), "flip_fraction": frac,
                    "max_ulps": int(ulps.max()) if ulps.size else 0}
    bad = np.nonzero(~inside.reshape(-1))[0]
    assert bad.size == 0, (f"{name}: {bad.size} elements outside the float32 error bound, e.g. flat index {bad[:5]}: "
                           f"gpu {g.reshape(-1)[bad[:5]]}, exact {exact.reshape(-1)[bad[:5]]}, "
                           f"bound {E.reshape(-1)[bad[:5]]}")
    # more than one ulp only where the float32 bound itself spans more than half an ulp (values near zero
    # after cancellation in a sum, whose bf16 ulp is far below the sum's rounding error)
    ulp = np.ldexp(1.0, np.frexp(np.maximum(np.abs(exact), 1e-300))[1] - 8)
    wide = ulps > 1
    report[name]["beyond_one_ulp"] = int(wide.sum())
    assert not (wide & (E < 0.5 * ulp)).any(), \
        f"{name}: {int((wide & (E < 0.5 * ulp)).sum())} elements more than one bf16 ulp off where the bound is below half an ulp"
    assert frac <= max_flip, f"{name}: rounding flips in {frac:.4f} of the elements"


def check_f32(name, gpu, exact, E, report):
    """GPU float32 output vs the exact stage value: |gpu - exact| <= E element by element."""
    exact = np.asarray(exact, np.float64)
    d = np.abs(np.asarray(gpu, np.float64).reshape(exact.shape) - exact)
    E = np.broadcast_to(np.asarray(E, np.float64), exact.shape)
    ratio = d / np.maximum(E, 1e-300)
    report[name] = {"elements": int(d.size), "max_abs": float(d.max()) if d.size else 0.0,
                    "max_ratio_to_bound": float(ratio.max()) if d.size else 0.0,
                    "median_ratio_to_bound": float(np.median(ratio)) if d.size else 0.0}
    bad = np.nonzero((d > E).reshape(-1))[0]
    assert bad.size == 0, (f"{name}: {bad.size} elements beyond the float32 error bound, e.g. flat index {bad[:5]}: "
                           f"|diff| {d.reshape(-1)[bad[:5]]}, bound {E.reshape(-1)[bad[:5]]}")


# ---------------------------------------------------------------- per-stage float32 error bounds

def norm_bound(exact_u_unrounded, d):
    """RMSNorm u = r g / sqrt(mean(r^2) + eps): the sum of d squares (gamma_{d+2} relative, all terms
    positive), square root and reciprocal (a relative error of half that plus a few ulps), two products."""
    return (0.5 * gamma(d + 2) + 8 * U) * np.abs(exact_u_unrounded)


def linear_bound(x_abs, w_abs, bias_abs=None, extra_terms=0):
    """|fl(x w^T + b) - (x w^T + b)| <= gamma_{K+1+extra} (|x| |w|^T + |b|)."""
    K = x_abs.shape[-1]
    s = x_abs @ w_abs.T
    if bias_abs is not None:
        s = s + bias_abs
    return gamma(K + 1 + extra_terms) * s


def rope_pair_bound(E_pre, pre, half):
    """Rotation (a, b) -> (a cos - b sin, b cos + a sin) with |cos|, |sin| <= 1 from a float32 table:
    the error of either output is at most E_a + E_b + 5 U (|a| + |b|). Arrays [..., dh]."""
    Ea, Eb = E_pre[..., :half], E_pre[..., half:]
    a, b = np.abs(pre[..., :half]), np.abs(pre[..., half:])
    e = Ea + Eb + 5 * U * (a + b)
    return np.concatenate([e, e], axis=-1)


def attention_bound(q, k, v, P, scale_log2):
    """Softmax attention o = sum_j P_j v_j evaluated in float32 with scores s_j = q.k_j, probabilities
    exp2(s_j * scale - m) normalised at the end. Per query row and output dimension (first order):
    |do| <= 2 H sum_j P_j |v_j| + (2 gamma_{Sk+4} + 2 U) sum_j P_j |v_j|, where H bounds the relative
    error of any unnormalised probability: ln 2 (scale eps_j + 4 U (|t_j| + max|t|)) + 2^-21 with
    eps_j = gamma_{dh} sum_d |q_d k_jd| and t_j = s_j * scale (log2 units).
    q [Sq, dh], k and v [Sk, dh], P [Sq, Sk] (the exact probabilities); returns [Sq, dh]."""
    dh = q.shape[-1]
    Sk = k.shape[0]
    eps = gamma(dh) * (np.abs(q) @ np.abs(k).T)                 # [Sq, Sk]
    t = np.abs(q @ k.T) * scale_log2
    H = np.log(2.0) * (scale_log2 * eps + 4 * U * (t + t.max(axis=1, keepdims=True))) + 2.0 ** -21
    w = P @ np.abs(v)                                            # sum_j P_j |v_j|, [Sq, dh]
    return (2 * H.max(axis=1, keepdims=True) + 2 * gamma(Sk + 4) + 2 * U) * w * 1.01


def swiglu_bound(g, up, Eg, Eu):
    """a = silu(g) up with |silu'| <= 1.1: 1.1 Eg |up| + |silu(g)| Eu + Eg Eu, plus the float32 evaluation of
    silu(g) up itself (exp of -g through exp2 with a rounded argument: (|g| + 8) U + 2^-22 relative)."""
    s = g / (1.0 + np.exp(-g))
    a = s * up
    return 1.1 * Eg * np.abs(up) + np.abs(s) * Eu + Eg * Eu + ((np.abs(g) + 8) * U + 2.0 ** -22) * np.abs(a)
