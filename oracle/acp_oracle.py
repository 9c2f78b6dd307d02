"""Dense float64 reference for Forgetting Attention with ACP (one head at a time).

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the benchmark's
CPU-baseline leg, never by the product path.

Indices are 0-based here; the paper's are 1-based.  The pruning grid uses square
blocks of BLOCK = 64 rows by 64 columns.

Every function cites the passage of the paper it follows.  Points where the paper
is silent or garbled are settled as follows (the same readings bind the HIP path):

* cumulative gates (Sec. 2, "FlashAttention implementation"): c_i is the float32
  rounding (to nearest, ties to even) of the exact sum of log f_l for l <= i.
  Being the rounding of an exact value, it does not depend on the order of the
  additions, so a parallel scan can reproduce it bit for bit; c is the canonical
  float32 quantity both sides compare on.
* logit bound (Sec. 3, "Safe pruning"): U = rho_q * rho_k / sqrt(d), with rho the
  largest row L2 norm of the stored Q (resp. K) of the one sequence and head.
  Squared norms are float64 sums in ascending feature order; U = sqrt(rq2*rk2/d)
  with IEEE round-to-nearest float64 operations.
* threshold (Sec. 3, eq. for delta; App. A): delta = -(2U + (log L - log eps)),
  natural logarithms, L the full context length, float64.  eps = 0 gives
  delta = -inf (nothing pruned).
* block rule (Sec. 3, "Block-level pruning"): block (m, n) is pruned iff every
  causal entry of D in it is below delta (strict), decided in float64 on the
  float32 c.  Diagonal blocks always hold D_ii = 0 and are kept.
* Algorithm 1 as printed assigns the boundary index after incrementing past the
  first kept block; the reading used here is "first kept block of the row"
  (the boundary block the text defines), so the pointer is tested before it is
  advanced.
* decoding (App. F): the bound U must be known before the tokens are (QK-norm
  scales, App. E), and the threshold is sized for the longest sequence L_max,
  delta = -(2U + log L_max - log eps), so that it stays fixed as t grows (App. A
  needs only that a row holds at most L_max entries).  A cache of fixed size
  keeps the last positions; see decode_ring_row for what is attended when it
  has dropped a kept key.
* backward: the paper only says it follows the forward.  The mask is a constant
  (the indicator has zero derivative almost everywhere, and delta's dependence on
  Q and K is not differentiated).  With x_ij = q_i.k_j/sqrt(d) + c_i - c_j:
  dS = P o (dP - Delta), dQ = dS K / sqrt(d), dK = dS^T Q / sqrt(d),
  dc = rowsum(dS) - colsum(dS), and dlog f_l = sum_{i >= l} dc_i.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

BLOCK = 64

__all__ = [
    "BLOCK", "cumsum_log_gates", "cumsum_exact_fraction", "cumsum_span_bits",
    "cumsum_inexact_flag", "gate_logits", "log_sigmoid", "gate_log_forget",
    "row_norm_sq_max", "logit_bound", "logit_bound_qknorm", "log_len_over_eps", "threshold",
    "entry_keep", "block_keep_bruteforce", "block_keep_topright", "boundary_from_block_keep",
    "boundary_alg1", "col_end_from_row_start", "kept_tiles", "causal_tiles",
    "block_mask", "entry_mask", "causal_mask", "forward", "backward", "pruned_mass",
    "plan_head", "run_head", "forward_rows", "backward_rows", "backward_cols",
    "backward_row_range",
    "decode_pointer", "decode_row", "decode_ring_row", "qk_projection",
]


# --------------------------------------------------------------------------
# Stage 1: cumulative log gates, logit bound, threshold, boundary
# --------------------------------------------------------------------------

def cumsum_log_gates(log_f) -> np.ndarray:
    """c_i = sum_{l<=i} log f_l (Sec. 2, FlashAttention paragraph: D = c1^T - 1c^T).

    The float32 rounding of the exact prefix sum of the float32 gates.  Where a
    row's partial sums span at most 53 bits (cumsum_span_bits) every float64
    running sum is exact, and one rounding of it gives c; wider rows are summed
    exactly in integers.  A sum beyond the float32 range rounds to -inf.
    """
    x = np.asarray(log_f, dtype=np.float32)
    flat = x.reshape(-1, x.shape[-1]) if x.ndim else x.reshape(1, 1)
    out = np.empty(flat.shape, dtype=np.float32)
    for r in range(flat.shape[0]):
        row = flat[r]
        if not np.all(np.isfinite(row)) or cumsum_span_bits(row) <= 53:
            acc = np.cumsum(row.astype(np.float64))
            # a sum beyond the float32 range rounds to -inf (IEEE round-to-nearest),
            # which is the value the checks expect; numpy would only warn about it
            with np.errstate(over="ignore", invalid="ignore"):
                out[r] = acc.astype(np.float32)
        else:
            out[r] = _exact_prefix_f32(row)
    return out.reshape(x.shape)


def _exact_prefix_f32(row) -> np.ndarray:
    """Prefix sums of finite float32 values, exact in integers (each value is an
    integer significand times a power of two), each rounded once to float32."""
    f, e = np.frexp(np.asarray(row, dtype=np.float32).astype(np.float64))
    m = (f * 2.0 ** 24).astype(np.int64)          # exact: at most 24 significant bits
    k = e.astype(np.int64) - 24                   # row[i] = m[i] * 2^k[i]
    nz = m != 0
    out = np.zeros(len(m), dtype=np.float32)
    if not nz.any():
        return out
    lsb = int(k[nz].min())
    acc = 0
    for i in range(len(m)):
        if m[i]:
            acc += int(m[i]) << int(k[i] - lsb)
        out[i] = _int_to_f32(acc, lsb)
    return out


def _int_to_f32(n: int, lsb: int) -> np.float32:
    """Round n * 2^lsb (n an integer) to the nearest float32, ties to even."""
    if n == 0:
        return np.float32(0.0)
    sign = -1.0 if n < 0 else 1.0
    a = abs(n)
    e = max(a.bit_length() - 1 + lsb, -126)       # 2^e <= |value| < 2^(e+1); subnormals at -126
    shift = (e - 23) - lsb                        # drop bits below 2^(e-23)
    if shift <= 0:
        q = a << -shift
    else:
        q, rem = a >> shift, a & ((1 << shift) - 1)
        half = 1 << (shift - 1)
        if rem > half or (rem == half and q & 1):
            q += 1
    if e - 23 > 104 or (e - 23 == 104 and q >= 1 << 24):
        return np.float32(sign * np.inf)         # beyond the largest float32
    return np.float32(sign * math.ldexp(float(q), e - 23))


def gate_logits(x, w_f, b_f) -> np.ndarray:
    """Forget-gate logits a_t = w_f^T x_t + b_f of every head (Sec. 2: each head's
    gate is f_t = sigmoid(w_f^T x_t + b_f) of the layer input x_t).

    x [T, d_model] and w_f [d_model, H] are bfloat16 values, b_f [H] float32.
    Reading (the paper does not fix the precision): the dot product is summed in
    float32 in ascending feature order, each step one rounding (a product of two
    bfloat16 values is exact in float32), and b_f is added last, in float32.
    Returns [T, H] float32.
    """
    x32 = np.asarray(x, dtype=np.float32)
    w32 = np.asarray(w_f, dtype=np.float32)
    acc = np.zeros((x32.shape[0], w32.shape[1]), dtype=np.float32)
    for k in range(x32.shape[1]):
        acc = acc + x32[:, k:k + 1] * w32[k:k + 1, :]
    return acc + np.asarray(b_f, dtype=np.float32)[None, :]


def log_sigmoid(a) -> np.ndarray:
    """log f = log sigmoid(a) = -softplus(-a) (Sec. 2 gate), in float64 as
    -(max(-a, 0) + log1p(exp(-|a|))), rounded once to float32."""
    a64 = np.asarray(a, dtype=np.float32).astype(np.float64)
    return (-(np.maximum(-a64, 0.0) + np.log1p(np.exp(-np.abs(a64))))).astype(np.float32)


def gate_log_forget(x, w_f, b_f, B: int) -> np.ndarray:
    """log f [B, H, L] of a layer input x [B*L, d_model] (token l of sequence b is
    row b*L + l): log_sigmoid(gate_logits(x, w_f, b_f))."""
    lf = log_sigmoid(gate_logits(x, w_f, b_f))
    T, H = lf.shape
    return np.ascontiguousarray(lf.reshape(B, T // B, H).transpose(0, 2, 1))


def cumsum_exact_fraction(log_f_1d) -> np.ndarray:
    """Exact rational prefix sums of float32 values, each rounded once to float32.

    An independent definition of the canonical c (used to pin cumsum_log_gates).
    """
    vals = [Fraction(float(v)) for v in np.asarray(log_f_1d, dtype=np.float32)]
    out = np.empty(len(vals), dtype=np.float32)
    acc = Fraction(0)
    for i, v in enumerate(vals):
        acc += v
        out[i] = _fraction_to_f32(acc)
    return out


def _fraction_to_f32(fr: Fraction) -> np.float32:
    """Round an exact rational to the nearest float32, ties to even (one rounding)."""
    if fr == 0:
        return np.float32(0.0)
    sign = -1 if fr < 0 else 1
    a = abs(fr)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1                                  # now 2^e <= a < 2^(e+1)
    e = max(e, -126)                            # subnormals share the lowest exponent
    scaled = a * Fraction(2) ** (23 - e)        # 24-bit significand in [2^23, 2^24)
    n, rem = divmod(scaled.numerator, scaled.denominator)
    twice = 2 * rem
    if twice > scaled.denominator or (twice == scaled.denominator and n % 2 == 1):
        n += 1
    return np.float32(sign * math.ldexp(float(n), e - 23))


def cumsum_span_bits(log_f_1d) -> int:
    """Bits spanned by the partial sums of float32 addends (0 if all are zero).

    Every float32 addend is an integer multiple of 2^lsb, lsb = e_min - 23 the
    exponent of the smallest ulp among the nonzero addends (subnormals share the
    smallest normal exponent), and every partial sum lies below 2^E, the least
    power of two above the exact sum of |x|.  Such a value needs at most E - lsb
    significant bits, so when E - lsb <= 53 all float64 partial sums are exact and
    any summation order gives the same c.  The total is summed exactly (fsum
    rounds once, to nearest, and so is below 2^E exactly when the exact sum is).
    """
    x = np.asarray(log_f_1d, dtype=np.float32).astype(np.float64)
    nz = x[x != 0]
    if nz.size == 0:
        return 0
    _, e = np.frexp(np.abs(nz))          # |x| = m * 2^e, m in [0.5, 1)
    lsb = int(np.min(np.maximum(e - 1, -126))) - 23
    total = math.fsum(np.abs(nz).tolist())
    E = math.frexp(total)[1]             # 2^(E-1) <= total < 2^E
    return E - lsb


def cumsum_inexact_flag(log_f_1d) -> bool:
    """Flag bit 2 of stage 1 (reading of Sec. 2's cumulative sum, whose precision
    the paper leaves open): raised when the span is 105 bits or more.  The device
    sums in double-double (pairs of float64 values), which is exact for any
    association while the span is at most 105 bits; its double-double sum of |x|
    is then exact too, so it reads every span up to 105 exactly and wider ones as
    at least 105.  Clear, the flag guarantees that c is the rounding of the exact
    sum."""
    return cumsum_span_bits(log_f_1d) >= 105


def row_norm_sq_max(x) -> float:
    """rho^2 = max_i sum_k x_ik^2 (Sec. 3, 'we can set U = rho_q rho_k / sqrt(d)').

    x is [L, d]; the squared norm of each row is a float64 sum in ascending k.
    """
    x = np.asarray(x, dtype=np.float64)
    acc = np.zeros(x.shape[0], dtype=np.float64)
    for kk in range(x.shape[1]):
        acc = acc + x[:, kk] * x[:, kk]
    return float(np.max(acc)) if acc.size else 0.0


def logit_bound(rho2_q: float, rho2_k: float, d: int) -> float:
    """U = rho_q rho_k / sqrt(d), evaluated as sqrt(rho_q^2 rho_k^2 / d) (Sec. 3)."""
    return math.sqrt((float(rho2_q) * float(rho2_k)) / float(d))


def logit_bound_qknorm(gamma_q: float, gamma_k: float, d: int) -> float:
    """U from QK-norm scales (App. E; Sec. 3 allows any valid bound on the logits):
    an RMS-normalised row has norm sqrt(d), an elementwise scale of magnitude at
    most gamma multiplies that by at most gamma, so |q.k| / sqrt(d) is at most
    gamma_q sqrt(d) gamma_k sqrt(d) / sqrt(d) = gamma_q gamma_k sqrt(d).  The scales
    are float32; their product is exact in float64; one rounding per operation."""
    gq = float(np.float32(gamma_q))
    gk = float(np.float32(gamma_k))
    return (gq * gk) * math.sqrt(d)


def log_len_over_eps(L: int, eps: float) -> float:
    """log L - log eps (natural logs, Sec. 3 and App. A); +inf for eps = 0."""
    if eps == 0.0:
        return math.inf
    return math.log(float(L)) - math.log(float(eps))


def threshold(U: float, L: int, eps: float) -> float:
    """delta = -2U - log L + log eps (Sec. 3, 'Safe pruning'; proof in App. A)."""
    return -(2.0 * U + log_len_over_eps(L, eps))


def entry_keep(c, delta: float) -> np.ndarray:
    """keep_ij = (j <= i) and D_ij >= delta with D_ij = c_i - c_j (Sec. 3, eq. 3)."""
    c64 = np.asarray(c, dtype=np.float32).astype(np.float64)
    L = c64.shape[0]
    D = c64[:, None] - c64[None, :]
    return np.tril(np.ones((L, L), dtype=bool)) & (D >= delta)


def block_keep_bruteforce(c, delta: float, block: int = BLOCK) -> np.ndarray:
    """Keep_mn = some causal entry of block (m, n) has D_ij >= delta (Sec. 3, block-level).

    Decided entry by entry; diagonal blocks contain D_ii = 0 and so are kept
    whenever delta <= 0 (footnote of the block-level paragraph).
    """
    keep = entry_keep(c, delta)
    L = keep.shape[0]
    M = L // block
    kb = keep.reshape(M, block, M, block).any(axis=(1, 3))
    kb[np.arange(M), np.arange(M)] = True
    return kb


def block_keep_topright(c, delta: float, block: int = BLOCK) -> np.ndarray:
    """Keep_mn decided on the top-right entry of each block (Sec. 3, block-level paragraph).

    For n < m the largest entry of D[m][n] is c_{block*m} - c_{block*n + block-1}
    by coordinate-wise monotonicity (Sec. 2).  Blocks above the diagonal are not
    causal; diagonal blocks are kept.
    """
    c64 = np.asarray(c, dtype=np.float32).astype(np.float64)
    M = c64.shape[0] // block
    first = c64[np.arange(M) * block]
    last = c64[np.arange(M) * block + block - 1]
    kb = (first[:, None] - last[None, :]) >= delta
    kb &= np.tril(np.ones((M, M), dtype=bool))
    kb[np.arange(M), np.arange(M)] = True
    return kb


def boundary_from_block_keep(kb: np.ndarray):
    """row_start[m] = min{n: Keep_mn}, col_end[n] = max{m: Keep_mn} (Sec. 3, two-stage)."""
    M = kb.shape[0]
    row_start = np.array([int(np.argmax(kb[m, :m + 1])) for m in range(M)], dtype=np.int32)
    col_end = np.array([n + int(np.nonzero(kb[n:, n])[0].max()) for n in range(M)],
                       dtype=np.int32)
    return row_start, col_end


def boundary_alg1(c, delta: float, block: int = BLOCK) -> np.ndarray:
    """Linear-time boundary search (Sec. 3, Algorithm 1), first-kept-block reading.

    One pointer l walks the key blocks; for each query block m it advances while
    the top-right entry of block (m, l) is below delta, and never moves back.
    """
    c64 = np.asarray(c, dtype=np.float32).astype(np.float64)
    M = c64.shape[0] // block
    out = np.empty(M, dtype=np.int32)
    l = 0
    for m in range(M):
        while l < m and (c64[block * m] - c64[block * l + block - 1]) < delta:
            l += 1
        out[m] = l
    return out


def col_end_from_row_start(row_start) -> np.ndarray:
    """Column form of the staircase: col_end[n] = max{m : row_start[m] <= n}."""
    rs = np.asarray(row_start)
    M = rs.shape[0]
    return np.array([max(m for m in range(M) if rs[m] <= n) for n in range(M)], dtype=np.int32)


def kept_tiles(row_start) -> int:
    rs = np.asarray(row_start, dtype=np.int64)
    return int(np.sum(np.arange(rs.shape[0]) - rs + 1))


def causal_tiles(M: int) -> int:
    """Causal 64x64 blocks of one head, M(M+1)/2 (denominator of the pruned fraction)."""
    return M * (M + 1) // 2


# --------------------------------------------------------------------------
# Masks
# --------------------------------------------------------------------------

def causal_mask(L: int) -> np.ndarray:
    return np.tril(np.ones((L, L), dtype=bool))


def block_mask(row_start, L: int, block: int = BLOCK) -> np.ndarray:
    """Mask_ij = (j <= i) and block (i//block, j//block) is kept (block-level ACP)."""
    rs = np.asarray(row_start)
    qb = np.arange(L) // block
    kb = np.arange(L) // block
    return causal_mask(L) & (kb[None, :] >= rs[qb][:, None])


def entry_mask(c, delta: float) -> np.ndarray:
    """Entry-level ACP mask of eq. 3."""
    return entry_keep(c, delta)


# --------------------------------------------------------------------------
# Stage 2: attention forward / backward (dense, float64)
# --------------------------------------------------------------------------

def _logits(q, k, c, mask):
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    c64 = np.asarray(c).astype(np.float64)
    d = q.shape[1]
    s = (q @ k.T) / math.sqrt(d)
    x = s + (c64[:, None] - c64[None, :])
    return np.where(mask, x, -np.inf)


def forward(q, k, v, c, mask):
    """O = softmax(Q K^T / sqrt(d) + D) V restricted to `mask`, and the row log-sum-exp.

    Sec. 2, eq. 1-2 (Forgetting Attention), with the ACP indicator of eq. 3 folded
    into `mask` (block-level mask for the pruned kernel, causal mask for eq. 1).
    Returns (O [L,d] float64, LSE [L] float64).
    """
    x = _logits(q, k, c, mask)
    m = np.max(x, axis=1, keepdims=True)
    e = np.exp(x - m)
    z = np.sum(e, axis=1, keepdims=True)
    p = e / z
    o = p @ np.asarray(v, dtype=np.float64)
    lse = (m + np.log(z))[:, 0]
    return o, lse


def backward(q, k, v, c, mask, do, o=None, lse=None):
    """Gradients of the masked forward (the paper says only that the backward mirrors
    the forward, Sec. 2; formulas derived by the chain rule through eq. 2 and c).

    Returns a dict with dq, dk, dv, dlog_f ([L]) and the intermediates dS, dc.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    d = q.shape[1]
    if o is None or lse is None:
        o, lse = forward(q, k, v, c, mask)
    x = _logits(q, k, c, mask)
    p = np.exp(x - lse[:, None])
    dv = p.T @ do
    dp = do @ v.T
    delta_row = np.sum(do * o, axis=1)
    ds = p * (dp - delta_row[:, None])
    dq = (ds @ k) / math.sqrt(d)
    dk = (ds.T @ q) / math.sqrt(d)
    dc = np.sum(ds, axis=1) - np.sum(ds, axis=0)
    dlog_f = np.cumsum(dc[::-1])[::-1].copy()
    return {"dq": dq, "dk": dk, "dv": dv, "dlog_f": dlog_f, "ds": ds, "dc": dc,
            "o": o, "lse": lse}


def pruned_mass(q, k, c, kept_mask):
    """Per row, the total full-attention weight (eq. 1) that `kept_mask` drops (App. A)."""
    L = np.asarray(q).shape[0]
    full = causal_mask(L)
    x = _logits(q, k, c, full)
    m = np.max(x, axis=1, keepdims=True)
    a = np.exp(x - m)
    a /= np.sum(a, axis=1, keepdims=True)
    return np.sum(np.where(full & ~kept_mask, a, 0.0), axis=1)


# --------------------------------------------------------------------------
# One head end to end
# --------------------------------------------------------------------------

def plan_head(q, k, log_f, eps: float, block: int = BLOCK, method: str = "bruteforce",
              U: float | None = None):
    """Stage 1 for one (batch, head): c, U, delta and the boundary (Sec. 3).  A given
    U (e.g. logit_bound_qknorm) replaces the bound from the row norms."""
    L, d = np.asarray(q).shape
    c = cumsum_log_gates(log_f)
    if U is None:
        rq = row_norm_sq_max(q)
        rk = row_norm_sq_max(k)
        U = logit_bound(rq, rk, d)
    else:
        rq = rk = float("nan")
    delta = threshold(U, L, eps)
    if method == "bruteforce":
        kb = block_keep_bruteforce(c, delta, block)
        row_start, col_end = boundary_from_block_keep(kb)
    elif method == "topright":
        kb = block_keep_topright(c, delta, block)
        row_start, col_end = boundary_from_block_keep(kb)
    elif method == "alg1":
        row_start = boundary_alg1(c, delta, block)
        col_end = col_end_from_row_start(row_start)
    else:
        raise ValueError(method)
    return {"c": c, "rho2_q": rq, "rho2_k": rk, "U": U, "delta": delta,
            "row_start": row_start, "col_end": col_end, "kept": kept_tiles(row_start)}


def run_head(q, k, v, log_f, eps: float, do=None, block: int = BLOCK, method: str = "topright",
             U: float | None = None):
    """Plan, pruned forward and (if do is given) backward for one head (U: as in
    plan_head)."""
    plan = plan_head(q, k, log_f, eps, block, method, U)
    L = np.asarray(q).shape[0]
    mask = block_mask(plan["row_start"], L, block)
    o, lse = forward(q, k, v, plan["c"], mask)
    out = dict(plan)
    out.update({"o": o, "lse": lse, "mask": mask})
    if do is not None:
        g = backward(q, k, v, plan["c"], mask, do, o, lse)
        out.update({kk: g[kk] for kk in ("dq", "dk", "dv", "dlog_f", "dc")})
    return out


# --------------------------------------------------------------------------
# Selected rows / columns of the same dense definition (for long sequences,
# where the full L x L matrices of every head are too large to form)
# --------------------------------------------------------------------------

def _row_logits(q, k, c, row_start, i, block: int = BLOCK):
    """Masked logits of query row i (eq. 2 with the block-level ACP mask)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    c64 = np.asarray(c).astype(np.float64)
    d = q.shape[1]
    j = np.arange(i + 1)
    keep = (j // block) >= int(row_start[i // block])
    x = (k[: i + 1] @ q[i]) / math.sqrt(d) + (c64[i] - c64[: i + 1])
    return np.where(keep, x, -np.inf)


def forward_rows(q, k, v, c, row_start, rows, block: int = BLOCK):
    """O and LSE of the pruned forward for the query rows `rows` (Sec. 2 eq. 1; each
    row of eq. 1 depends only on its own logits).  Returns (O [n,d], LSE [n])."""
    v = np.asarray(v, dtype=np.float64)
    o = np.empty((len(rows), v.shape[1]))
    lse = np.empty(len(rows))
    for r, i in enumerate(rows):
        x = _row_logits(q, k, c, row_start, i, block)
        m = np.max(x)
        e = np.exp(x - m)
        z = np.sum(e)
        o[r] = (e / z) @ v[: i + 1]
        lse[r] = m + math.log(z)
    return o, lse


def backward_rows(q, k, v, c, row_start, do, rows, block: int = BLOCK):
    """dQ and rowsum(dS) for the query rows `rows` (chain rule as in `backward`; a
    row of dQ needs only that row of dS).  Returns (dQ [n,d], rowsum [n])."""
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    d = k.shape[1]
    dq = np.empty((len(rows), d))
    rs = np.empty(len(rows))
    for r, i in enumerate(rows):
        x = _row_logits(q, k, c, row_start, i, block)
        p = np.exp(x - np.max(x))
        p /= np.sum(p)
        o_i = p @ v[: i + 1]
        dp = v[: i + 1] @ do[i]
        ds = p * (dp - do[i] @ o_i)
        dq[r] = (ds @ k[: i + 1]) / math.sqrt(d)
        rs[r] = np.sum(ds)
    return dq, rs


def backward_cols(q, k, v, c, row_start, do, cols, block: int = BLOCK):
    """dK, dV and colsum(dS) for the key columns `cols`: column j collects dS_ij and
    P_ij over every query row i >= j whose block keeps it, each row normalised by
    its own softmax.  Returns (dK [n,d], dV [n,d], colsum [n])."""
    q = np.asarray(q, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    L, d = q.shape
    rs = np.asarray(row_start)
    dk = np.zeros((len(cols), d))
    dv = np.zeros((len(cols), d))
    cs = np.zeros(len(cols))
    for r, j in enumerate(cols):
        for i in range(j, L):
            if (j // block) < int(rs[i // block]):
                continue
            x = _row_logits(q, k, c, rs, i, block)
            p = np.exp(x - np.max(x))
            p /= np.sum(p)
            o_i = p @ v[: i + 1]
            dp_ij = do[i] @ v[j]
            ds_ij = p[j] * (dp_ij - do[i] @ o_i)
            dv[r] += p[j] * do[i]
            dk[r] += ds_ij * q[i] / math.sqrt(d)
            cs[r] += ds_ij
    return dk, dv, cs


def backward_row_range(q, k, v, c, row_start, do, r0: int, r1: int, ls=(), group: int = 256,
                       block: int = BLOCK):
    """The dense definition of `forward` / `backward` evaluated for the query rows
    r0 <= i < r1 only, a group of rows at a time, so that a long head never needs
    its L x L matrices at once.  Each row's softmax is taken over its own kept keys
    (eq. 2 with the block-level mask of Sec. 3; a row depends on no other row), and
    its gradient terms follow the chain rule of `backward`.

    Returns o, lse, dq, rowsum for rows r0..r1-1, and, summed over those rows only,
    dk, dv ([L, d]) and colsum ([L]); these are the full column values for every
    key j all of whose keeping rows lie in the range (rows i >= j of the blocks up
    to col_end of j's block).  rect[l] for each l in `ls` is the part of the
    rectangle identity dlog f_l = sum_{i >= l} sum_{j < l} dS_ij that these rows
    hold (all of it when the range covers every row >= l that keeps a key < l).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    c64 = np.asarray(c).astype(np.float64)
    rs = np.asarray(row_start)
    L, d = q.shape
    sd = math.sqrt(d)
    n = r1 - r0
    out = {"o": np.empty((n, d)), "lse": np.empty(n), "dq": np.empty((n, d)),
           "rowsum": np.empty(n), "dk": np.zeros((L, d)), "dv": np.zeros((L, d)),
           "colsum": np.zeros(L), "rect": {int(l): 0.0 for l in ls}}
    for g0 in range(r0, r1, group):
        rows = np.arange(g0, min(g0 + group, r1))
        lo = block * int(rs[rows[0] // block])        # the boundary only moves right
        hi = int(rows[-1]) + 1
        j = np.arange(lo, hi)
        keep = (j[None, :] <= rows[:, None]) & ((j[None, :] // block) >= rs[rows // block][:, None])
        x = (q[rows] @ k[lo:hi].T) / sd + (c64[rows][:, None] - c64[lo:hi][None, :])
        x = np.where(keep, x, -np.inf)
        m = np.max(x, axis=1, keepdims=True)
        e = np.exp(x - m)
        z = np.sum(e, axis=1, keepdims=True)
        p = e / z
        o = p @ v[lo:hi]
        dp = do[rows] @ v[lo:hi].T
        delta_row = np.sum(do[rows] * o, axis=1)
        ds = p * (dp - delta_row[:, None])
        sl = slice(g0 - r0, g0 - r0 + len(rows))
        out["o"][sl] = o
        out["lse"][sl] = (m + np.log(z))[:, 0]
        out["dq"][sl] = (ds @ k[lo:hi]) / sd
        out["rowsum"][sl] = np.sum(ds, axis=1)
        out["dk"][lo:hi] += (ds.T @ q[rows]) / sd
        out["dv"][lo:hi] += p.T @ do[rows]
        out["colsum"][lo:hi] += np.sum(ds, axis=0)
        for l in out["rect"]:
            sel = rows >= l
            if np.any(sel) and l > lo:
                out["rect"][l] += float(np.sum(ds[sel][:, : l - lo]))
    return out


# --------------------------------------------------------------------------
# Decoding (App. F, inference-time ACP: a per-head boundary pointer that only moves
# forward, with the cache entries behind it dropped)
# --------------------------------------------------------------------------

def decode_pointer(c, t: int, delta: float, block: int = BLOCK) -> int:
    """First kept key block for the single query t: block n < t // block is kept iff
    some entry of it has D_tj = c_t - c_j >= delta (eq. 3 for one row); c is
    non-increasing, so that entry is the block's last key, 64 n + 63.  The block
    holding t is always kept (D_tt = 0).  Compared in float64 on the float32 c.

    Because c_t only falls as t grows, the pointer never moves back, and the keys
    before 64 * pointer can be dropped for every later query as well."""
    c64 = np.asarray(c).astype(np.float64)
    nb = t // block
    for n in range(nb):
        if c64[t] - c64[n * block + block - 1] >= delta:
            return n
    return nb


def _attend_range(q_t, k, v, c, t: int, lo: int):
    """Eq. 1-2 for the single query t over the keys j = lo .. t: (o [d], lse)."""
    q_t = np.asarray(q_t, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    c64 = np.asarray(c).astype(np.float64)
    d = q_t.shape[0]
    j = np.arange(lo, t + 1)
    x = (k[j] @ q_t) / math.sqrt(d) + (c64[t] - c64[j])
    m = np.max(x)
    e = np.exp(x - m)
    z = np.sum(e)
    return (e / z) @ v[j], m + math.log(z)


def decode_row(q_t, k, v, c, t: int, delta: float, block: int = BLOCK):
    """Output of query t over the keys kept for it alone (eq. 1-2 on the entries
    j in [64 n_t, t] with n_t = decode_pointer): (o [d], lse, n_t)."""
    n = decode_pointer(c, t, delta, block)
    o, lse = _attend_range(q_t, k, v, c, t, n * block)
    return o, lse, n


def decode_ring_row(q_t, k, v, c, t: int, delta: float, capacity: int, block: int = BLOCK):
    """Decoding from a cache that holds only the last `capacity` positions,
    t - capacity + 1 .. t.  App. F proposes dropping the entries behind the
    pointer; a cache of fixed size may also have to drop kept ones.  Reading
    used here: the query then attends to the kept keys still held,
    j in [max(64 n_t, t - capacity + 1), t], `lost` says whether a kept key was
    dropped, and the pointer reported is max(n_t, block of position
    t - capacity + 1), the first block whose test can still be made.
    Returns (o [d], lse, pointer, lost)."""
    n = decode_pointer(c, t, delta, block)
    first = t - capacity + 1
    lost = first > 0 and n * block < first
    o, lse = _attend_range(q_t, k, v, c, t, max(n * block, first, 0))
    return o, lse, max(n, first // block if first > 0 else 0), lost



# --------------------------------------------------------------------------
# Projection (Sec. 2: q_i = W_q x_i, k_i = W_k x_i), whose stored output the
# bound's row norms are taken from (Sec. 3)
# --------------------------------------------------------------------------

def qk_projection(x, w, B: int, H: int, d: int) -> np.ndarray:
    """Head-split projection X W in float64: token l of sequence b is row b L + l
    of X [B L, d_model], feature e of head h is column h d + e of W [d_model, H d];
    the result is [B, H, L, d] (the layout the attention takes its queries and
    keys in)."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    L = x.shape[0] // B
    y = x @ w
    return y.reshape(B, L, H, d).transpose(0, 2, 1, 3)
