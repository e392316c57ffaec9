"""FP8 (OCP e4m3) linear layers with tensor-wise or row-wise scales
(Section 3.5.2: linear-layer GEMMs in FP8 with tensor- or row-wise scalers,
normalisation in fp32).

Test infrastructure only (see the package docstring).

* e4m3: 1 sign, 4 exponent (bias 7), 3 mantissa bits; largest finite value
  1.75 * 2^8 = 448, smallest normal 2^-6, subnormals k * 2^-9; the code
  S.1111.111 is NaN and there are no infinities.  A real value is rounded to
  the nearest e4m3 value, ties to even, and magnitudes beyond 448 saturate
  to 448 (the quantiser never produces more than 448 * (1 + 2^-23)).
* Quantisation of X [rows, cols]: the scale s is amax / 448 over a row
  (row-wise) or over the matrix (tensor-wise), 1 where amax is 0, and the
  code of x is e4m3(x * (1 / s)) (multiplication by the reciprocal scale, as
  row-wise quantisers usually do).  Where floating point decides these
  integers, the oracle takes the decision in the accelerator's precision: s,
  1 / s and x * (1 / s) are fp32 operations (IEEE, correctly rounded), then
  rounded to e4m3 exactly.
* Linear layer: Y = act((dec(qA) dec(qW)^T) * sA * sW + b), evaluated
  exactly (float64) on the decoded values.
"""
import numpy as np

E4M3_MAX = 448.0


def e4m3_code(v):
    """Codes (uint8) of the e4m3 values nearest to v (ties to even,
    saturating at +-448); v finite."""
    v = np.asarray(v, np.float64)
    a = np.abs(v)
    code = np.zeros(v.shape, np.int64)
    normal = a >= 2.0 ** -6
    m, e = np.frexp(np.where(normal, a, 1.0))            # a = m 2^e, m in [0.5, 1)
    e = e - 1                                            # a = (2m) 2^e, 2m in [1, 2)
    q = np.rint(a * np.ldexp(1.0, 3 - e))                # 3 fraction bits: q in [8, 16]
    carry = q >= 16
    q = np.where(carry, 8, q)
    e = np.where(carry, e + 1, e)
    nc = (e + 7) * 8 + (q - 8)
    nc = np.where(e > 8, 0x7E, np.minimum(nc, 0x7E))     # saturate at 448
    code = np.where(normal, nc, np.rint(a * 512.0)).astype(np.int64)   # subnormals: k 2^-9
    sign = np.signbit(v).astype(np.int64) << 7
    return (code | sign).astype(np.uint8)


def e4m3_value(code):
    """Values (float64) of e4m3 codes (NaN for S.1111.111)."""
    c = np.asarray(code, np.int64)
    s = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    f = c & 7
    val = np.where(e == 0, f * 2.0 ** -9, (1.0 + f / 8.0) * np.ldexp(1.0, e - 7))
    val = np.where((c & 0x7F) == 0x7F, np.nan, val)
    return s * val


def quantize(x, rowwise=True):
    """(codes uint8 [rows, cols], scales fp32 [rows] or [1]) of a 2-D array of
    bf16 / fp32 values."""
    x32 = np.asarray(x, np.float64).astype(np.float32)
    ax = np.abs(x32)
    amax = ax.max(axis=1) if rowwise else np.array([ax.max()] if ax.size else [0.0], np.float32)
    amax = amax.astype(np.float32)
    s = np.where(amax > 0, amax / np.float32(E4M3_MAX), np.float32(1.0)).astype(np.float32)
    r = (np.float32(1.0) / s).astype(np.float32)
    rb = r[:, None] if rowwise else r[None, :1]
    return e4m3_code((x32 * rb).astype(np.float32)), s


def dequantize(codes, scales, rowwise=True):
    v = e4m3_value(codes)
    sc = np.asarray(scales, np.float64)
    return v * (sc[:, None] if rowwise else sc[0])


def linear_fp8(qa, sa, qw, sw, bias=None, relu=False):
    """act((dec(qa) dec(qw)^T) * sa * sw + bias) in float64; scales row-wise
    when they have one entry per row."""
    A = e4m3_value(qa)
    W = e4m3_value(qw)
    y = A @ W.T
    sa = np.asarray(sa, np.float64)
    sw = np.asarray(sw, np.float64)
    y = y * (sa[:, None] if sa.size == A.shape[0] and A.shape[0] > 1 else sa[0])
    y = y * (sw[None, :] if sw.size == W.shape[0] and W.shape[0] > 1 else sw[0])
    if bias is not None:
        y = y + np.asarray(bias, np.float64)
    return np.maximum(y, 0.0) if relu else y


# ---------------------------------------------------------------------------
# Accepted deviation of an accelerator's FP8 product (comparison rule).
ALIGN_BITS = 13          # fraction bits the fp8 matrix instruction keeps after alignment
UA = 2.0 ** -24          # fp32 unit roundoff


def linear_fp8_bound(qa, sa, qw, sw, bias=None, fast_accum=False, step=64, block=128):
    """Element-wise bound of |accelerator - linear_fp8(...)| (before any
    output rounding) when the contraction runs on a matrix instruction that
    adds ``step`` products and its incoming partial sum after aligning them
    to the largest exponent among them with ALIGN_BITS fraction bits (so
    each addend is off by less than 2^-ALIGN_BITS times the largest
    magnitude; the incoming partial sum's magnitude is bounded by the sum of
    |products| it holds): with fast_accum the partial sum is chained through
    the whole of K; without, it is chained only inside each ``block`` of K
    (every block starts from zero) and the blocks' sums are added in fp32.
    Worst case over signs; the largest product of a step is bounded by the
    step's largest |a| times its largest |w|."""
    A = np.abs(e4m3_value(qa))
    W = np.abs(e4m3_value(qw))
    M, K = A.shape
    N = W.shape[0]
    u = 2.0 ** -ALIGN_BITS
    err = np.zeros((M, N))
    run = np.zeros((M, N))                 # sum of |products| before this step
    chained = np.zeros((M, N))             # ... in the partial sum entering this step
    for k0 in range(0, K, step):
        if not fast_accum and k0 % block == 0:
            chained = np.zeros((M, N))
        a_s, w_s = A[:, k0:k0 + step], W[:, k0:k0 + step]
        m_s = a_s.max(1)[:, None] * w_s.max(1)[None, :]
        s_s = a_s @ w_s.T
        err += (step + 1) * u * np.maximum(chained, m_s)
        run += s_s
        chained += s_s
    sums = 1 if fast_accum else -(-K // block)
    err += (sums + 2) * UA * run            # fp32 adds of the blocks' sums
    sa = np.asarray(sa, np.float64)
    sw = np.asarray(sw, np.float64)
    sab = sa[:, None] if sa.size == M and M > 1 else sa[0]
    swb = sw[None, :] if sw.size == N and N > 1 else sw[0]
    y_abs = run * sab * swb + (np.abs(bias) if bias is not None else 0.0)
    return err * sab * swb + 3 * UA * y_abs  # + the two scale products and the bias add


def emulate_aligned_sum(products, c_in=0.0, bits=ALIGN_BITS):
    """One aligned addition as measured on the matrix instruction: every
    addend truncated toward zero to `bits` fraction bits of the largest
    exponent among them, then summed exactly (a model used only to check
    that linear_fp8_bound covers such arithmetic)."""
    v = np.append(np.asarray(products, np.float64), c_in)
    mx = np.abs(v).max()
    if mx == 0:
        return 0.0
    unit = np.ldexp(1.0, int(np.floor(np.log2(mx))) - bits)
    return float(np.sum(np.trunc(v / unit) * unit))
