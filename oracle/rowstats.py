"""Row normalisers and planning candidates (oracle side).

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.

The draft and target distributions are softmaxes of temperature-scaled logits
(Section 2.3: stochastic decoding at temperature T). The first pass scores
tree nodes by cumulative draft path log-probability over a pool of the
top-scoring tokens of each position (Section 3.1; Appendix B.3).

Precision contract shared with the HIP path (a reading: the paper states no
precision):
  invT = fl32(1/T);  a_v = fl32(x_v * invT)   (x are fp32 or bf16 logits)
  lse64 = m + ln sum_v exp(a_v - m) in binary64, m = max_v a_v
  lse32 = fl32(lse64)                          (canonical normaliser)
  lp_j  = fl32(a_{c_j} - lse32)                (planning log-probabilities)
  candidates c_j: the first K tokens by (logit desc, token id asc).
"""
import numpy as np

STATUS_NONFINITE = 1
STATUS_DEGENERATE_RESIDUAL = 2
STATUS_BUDGET_SHORT = 4


def inv_temperature(T):
    """fl32(1/T), the correctly rounded binary32 reciprocal."""
    T = np.float32(T)
    if not (np.isfinite(T) and T > 0):
        raise ValueError("temperature must be finite and > 0")
    return np.float32(1.0) / T


def scaled(x, invT):
    """a = fl32(x * invT) elementwise (binary32 product), returned as float64 values."""
    x32 = np.asarray(x, dtype=np.float32)
    return (x32 * np.float32(invT)).astype(np.float64)


def row_ok(a):
    """A row is usable when it has no NaN, no +inf and at least one finite entry."""
    a = np.asarray(a, dtype=np.float64)
    if np.isnan(a).any() or np.isposinf(a).any():
        return False
    return bool(np.isfinite(a).any())


def lse64(a):
    """Natural-log normaliser of one scaled row, in binary64 (max-shifted sum)."""
    a = np.asarray(a, dtype=np.float64)
    m = a.max()
    return float(m + np.log(np.sum(np.exp(a - m))))


def lse32(a):
    return np.float32(lse64(a))


def topk(x, K):
    """Indices of the first K entries by (value desc, index asc)."""
    x = np.asarray(x, dtype=np.float64)
    order = np.lexsort((np.arange(x.shape[0]), -x))
    return order[:K].astype(np.int64)


def draft_rowstats(draft_row, invT, K):
    """Per draft row: (ok, lse64, lse32, topk ids, topk lp as float32)."""
    a = scaled(draft_row, invT)
    if not row_ok(a):
        return False, np.nan, np.float32(np.nan), np.full(K, -1, np.int64), np.full(K, np.nan, np.float32)
    l64 = lse64(a)
    l32 = np.float32(l64)
    ids = topk(np.asarray(draft_row, dtype=np.float64), K)
    lp = (a[ids].astype(np.float32) - l32).astype(np.float32)
    return True, l64, l32, ids, lp


def probs(a, lse):
    """Probabilities exp(a_v - lse) in binary64."""
    return np.exp(np.asarray(a, dtype=np.float64) - float(lse))
