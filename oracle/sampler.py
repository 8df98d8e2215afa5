"""Speculative accept / residual resample with behavior log-probabilities.

The serving engine verifies k draft tokens per sequence with the target model
(Sec. 4.1, table of scaling controls: number of speculative tokens, zero disables)
at temperature 1.0 with no top-p/top-k (Sec. 5.3, Sec. 5.4), and records the
emitted token IDs with their behavior log-probabilities at generation time
(Sec. 4.2, Eq. 1). The accept rule itself is not printed in the paper; it is the
published speculative-sampling rule (Leviathan, Kalman & Matias 2023; Chen et
al. 2023): draft x_i ~ q_i is kept with probability min(1, p_{i-1}(x_i)/q_i(x_i));
on the first rejection a replacement is drawn from norm(max(0, p - q)); when all
k drafts pass, one bonus token is drawn from the last row p_k.

Numeric reading shared with the GPU path (every choice is listed in the design notes):
  * row j of sequence b: p_j = softmax(l[b, j, :]) at temperature 1, with
    m = max_t l_t and S = sum_t exp(l_t - m) defined in exact arithmetic; here
    float64.
  * draft x_i (i = 1..k) is judged by row i-1 with uniform u[b, i-1]: accept iff
    u * q_i(x_i) * S < exp(l_x - m)   (the test u < p/q without a division), strict <.
    q absent (greedy drafts) means q_i is one-hot at x_i.
  * the single extra uniform u[b, k] draws the final token (replacement or bonus)
    by an integer inverse CDF: R_t = floor(r_t * 2^62) with r the residual
    max(0, p - q) (or p for the bonus), Tot = sum R_t, target = (Tot *
    floor(u * 2^32)) >> 32, token = smallest j with sum_{t<=j} R_t > target. If the
    residual mass is zero the draw falls back to p with the same uniform.
  * out_logprobs[j] = (l[tok] - m) - ln S for the token emitted at row j.

For every decision the oracle also returns its relative margin, so that a
disagreement with another implementation can be classified as a near-tie (a
difference within the other side's rounding of S) rather than a bug.
"""
import numpy as np

TWO62 = float(2 ** 62)


def row_stats(l_rows):
    """m = max_t l_t and S = sum_t exp(l_t - m) of each row (last axis), float64."""
    l = np.asarray(l_rows, dtype=np.float32).astype(np.float64)
    m = l.max(axis=-1)
    S = np.exp(l - m[..., None]).sum(axis=-1)
    return m, S


def fixed_point_draw(r, u):
    """Inverse-CDF draws on the integer grid, one per row.
    r: [n, V] float64 >= 0 with row mass <= 1 (+ rounding); u: [n] float32 in [0, 1).
    Returns (index [n] int64 (-1 where the total mass is 0), Tot [n] uint64, margin [n]),
    margin = distance of the target to the nearest CDF boundary, relative to Tot."""
    R = np.floor(np.asarray(r, dtype=np.float64) * TWO62).astype(np.uint64)
    tot = R.sum(axis=1, dtype=np.uint64)
    u32 = np.floor(np.asarray(u, dtype=np.float32).astype(np.float64) * 2.0 ** 32).astype(np.uint64)
    # target = (Tot * U32) >> 32 without a 128-bit type: split Tot into 32-bit halves
    hi, lo = tot >> np.uint64(32), tot & np.uint64(0xFFFFFFFF)
    target = hi * u32 + ((lo * u32) >> np.uint64(32))
    c = np.cumsum(R, axis=1, dtype=np.uint64)
    above = c > target[:, None]
    j = np.argmax(above, axis=1)
    rows = np.arange(len(j))
    c_hi = c[rows, j].astype(np.float64)
    c_lo = np.where(j > 0, c[rows, np.maximum(j - 1, 0)], 0).astype(np.float64)
    t = target.astype(np.float64)
    totf = np.maximum(tot.astype(np.float64), 1.0)
    margin = np.minimum(t - c_lo + 1.0, c_hi - t) / totf
    j = np.where(tot > 0, j, -1)
    return j.astype(np.int64), tot, margin


def spec_accept(logits, draft_tokens, uniforms, draft_probs=None):
    """logits [B, k+1, V] f32; draft_tokens [B, k] int; uniforms [B, k+1] f32;
    draft_probs [B, k, V] f32 or None (one-hot q at the draft).

    Returns dict: tokens [B, k+1] int32 (-1 padded), n_accepted [B] int32,
    logprobs [B, k+1] float32 (NaN padded), accept_margin [B, k] (NaN where not
    tested), draw_margin [B]. Sequences are independent; the batch axis is only
    vectorised over."""
    logits = np.asarray(logits, dtype=np.float32)
    B, kp1, V = logits.shape
    k = kp1 - 1
    drafts = np.asarray(draft_tokens).reshape(B, k).astype(np.int64)
    u = np.asarray(uniforms, dtype=np.float32).reshape(B, kp1)
    q = None if draft_probs is None else np.asarray(draft_probs, dtype=np.float32)
    l = logits.astype(np.float64)
    m, S = row_stats(logits)                                   # [B, k+1]
    lnS = np.log(S)
    bi = np.arange(B)
    tokens = np.full((B, kp1), -1, dtype=np.int32)
    lps = np.full((B, kp1), np.nan, dtype=np.float32)
    acc_margin = np.full((B, k), np.nan)
    n = np.full(B, k, dtype=np.int64)
    alive = np.ones(B, dtype=bool)          # every draft so far accepted
    for i in range(1, k + 1):               # draft x_i is judged by row i-1
        row = i - 1
        x = drafts[:, row]
        ex = np.exp(l[bi, row, x] - m[:, row])
        qx = np.ones(B) if q is None else q[bi, row, x].astype(np.float64)
        lhs = u[:, row].astype(np.float64) * qx * S[:, row]
        accept = lhs < ex
        with np.errstate(divide="ignore", invalid="ignore"):
            mg = np.where(ex > 0, np.abs(lhs - ex) / ex, np.inf)
        acc_margin[alive, row] = mg[alive]
        keep = alive & accept
        tokens[keep, row] = x[keep]
        lps[keep, row] = ((l[keep, row, x[keep]] - m[keep, row]) - lnS[keep, row]).astype(np.float32)
        n[alive & ~accept] = i - 1
        alive = keep
    rejected = ~alive
    # final token: residual draw at the first rejection, else the bonus draw from p_k
    lf = l[bi, n]                                              # [B, V]
    p = np.exp(lf - m[bi, n][:, None]) / S[bi, n][:, None]
    qi = np.minimum(n, max(k - 1, 0))        # the rejecting row (unused where n == k)
    qrow = np.zeros((B, V))
    if k > 0 and q is None:
        qrow[bi, drafts[bi, qi]] = 1.0
    elif k > 0:
        qrow = q[bi, qi].astype(np.float64)
    r = np.where(rejected[:, None], np.maximum(0.0, p - qrow), p)
    j, tot, mg = fixed_point_draw(r, u[:, k])
    empty = tot == 0
    if empty.any():                                            # residual mass vanished
        j2, _, mg2 = fixed_point_draw(p[empty], u[empty, k])
        j[empty], mg[empty] = j2, mg2
    tokens[bi, n] = j
    lps[bi, n] = ((lf[bi, j] - m[bi, n]) - lnS[bi, n]).astype(np.float32)
    return {"tokens": tokens, "n_accepted": n.astype(np.int32), "logprobs": lps,
            "accept_margin": acc_margin, "draw_margin": mg}


# ------------------------------------------------------------- closed forms (for pins)

def softmax64(l):
    l = np.asarray(l, dtype=np.float64)
    e = np.exp(l - l.max())
    return e / e.sum()


def acceptance_prob(p, q):
    """Probability that a draft x ~ q is accepted against target p: sum_t min(p_t, q_t)."""
    return float(np.minimum(p, q).sum())


def expected_accepted(alphas):
    """E[n] for per-position acceptance probabilities alpha_1..alpha_k (drafts ~ q)."""
    tot, run = 0.0, 1.0
    for a in alphas:
        run *= a
        tot += run
    return tot
