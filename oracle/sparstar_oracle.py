"""SparSTAR CPU oracle: TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 NumPy statement of what the SparSTAR hot path computes,
written from the paper (arXiv 2608.10519, "SparSTAR", Section 5).  Only the test
suite, the smoke check and the benchmark's CPU-baseline leg may import it; the
product path (the HIP library and its Python binding) never does, and this
module shares no code with it.

Every function works on ONE (batch, head) pair with 2-D arrays `[L, D]`; callers
loop over batch and heads (the method treats them independently, Section 5.1).
Inputs are the exact float values of the bf16 tensors the GPU path reads,
widened to float64.

Pins (tests/test_oracle_*.py) tie each function to something other than itself:
brute-force pairwise block compatibility, closed-form keep/budget tables,
brute-force subset enumeration for top-k, torch's float64 scaled-dot-product
attention with the token mask of Eq. (7), and closed forms (Q = 0, V = 1, one
valid key).  No function is left "parity unpinned".
"""
from __future__ import annotations

import math

import numpy as np


# --------------------------------------------------------------------------
# Section 5.1: original-order block partition
# --------------------------------------------------------------------------
def num_blocks(length: int, b: int) -> int:
    """n = ceil(L / b): the number of contiguous b-token blocks (Section 5.1)."""
    return -(-int(length) // int(b))


def block_token_range(j: int, length: int, b: int) -> tuple[int, int]:
    """Token-index set B_j of block j, as the half-open range [j*b, min((j+1)*b, L)).

    Blocks follow the attention-kernel order and are NOT aligned to segment
    boundaries (Section 5.1)."""
    return j * b, min((j + 1) * b, length)


def partition(x: np.ndarray, b: int) -> np.ndarray:
    """Split `x` [L, D] into n = ceil(L/b) contiguous blocks [n, b, D].

    The final partial block is zero-padded to the nominal length b (Section 5.1)."""
    length, d = x.shape
    n = num_blocks(length, b)
    padded = np.zeros((n * b, d), dtype=np.float64)
    padded[:length] = x
    return padded.reshape(n, b, d)


def pool(x: np.ndarray, b: int) -> np.ndarray:
    """Block means  x_bar_i = b^-1 * sum_r x~_{i,r}  over the zero-padded block.

    The divisor is the nominal block length b even for a partial final block, so
    the pooled vector's magnitude scales with block occupancy (Section 5.1,
    paragraph on the aggregated score)."""
    return partition(np.asarray(x, dtype=np.float64), b).sum(axis=1) / b


# --------------------------------------------------------------------------
# Section 5.1 / Eq. (3)-(4): segment block sets, keep set, selectable set
# --------------------------------------------------------------------------
def segment_blocks(token_range: tuple[int, int], lk: int, b: int) -> set[int]:
    """J_seg = { j : B_j intersects I_seg }  (Section 5.1).

    A block that only partly overlaps the segment still belongs to it; the
    intersection test also covers segments that cross a block boundary."""
    begin, end = token_range
    out = set()
    for j in range(num_blocks(lk, b)):
        t0, t1 = block_token_range(j, lk, b)
        if max(t0, begin) < min(t1, end):
            out.add(j)
    return out


def keep_ranges_for_clip(clip: int, text: tuple[int, int], ref: tuple[int, int]) -> list[tuple[int, int]]:
    """The token ranges forced dense by Eq. (3).

    Clip 1 keeps the text and the final image-pyramid reference; clip c >= 2
    keeps the text only (its preceding-clip reference is ranked jointly with
    the current-scale blocks)."""
    if clip < 1:
        raise ValueError("clip index starts at 1")
    return [text, ref] if clip == 1 else [text]


def keep_blocks(keep: list[tuple[int, int]], lk: int, b: int) -> list[int]:
    """J_keep: union of the block sets of the forced ranges (Eq. 3), ascending."""
    out: set[int] = set()
    for r in keep:
        out |= segment_blocks(r, lk, b)
    return sorted(out)


def selectable_blocks(keep_set: list[int], lk: int, b: int) -> list[int]:
    """J_sel = {all key blocks} minus J_keep (Eq. 4), ascending."""
    ks = set(keep_set)
    return [j for j in range(num_blocks(lk, b)) if j not in ks]


# --------------------------------------------------------------------------
# Section 5.2 and the supplement's sparsity schedule: scale-wise densities
# --------------------------------------------------------------------------
def scale_densities(scale_lq: list[int], finest_rho: list[float]) -> list[float | None]:
    """rho_{c,s} for every scale s of one clip group, in generation order.

    The schedule assigns the given densities to the len(finest_rho) finest
    scales (the last ones, in order of increasing token count) and is a lookup
    by query length: every scale whose token count equals that of a sparsified
    scale gets that scale's density (scales with equal token counts share a
    density); all other scales stay dense (None).  Two sparsified scales with
    equal token counts but different densities contradict the lookup."""
    n = len(finest_rho)
    if n > len(scale_lq):
        raise ValueError("more densities than scales")
    table: dict[int, float] = {}
    for lq, rho in zip(scale_lq[len(scale_lq) - n:], finest_rho):
        if not (0.0 <= rho <= 1.0):
            raise ValueError("densities lie in [0, 1]")
        if table.get(lq, rho) != rho:
            raise ValueError("equal token counts with different densities")
        table[lq] = rho
    return [table.get(lq) for lq in scale_lq]


# --------------------------------------------------------------------------
# Eq. (5): the budget
# --------------------------------------------------------------------------
def budget_k(rho: float, n_sel: int) -> int:
    """k = min(n_sel, max(1, ceil(rho * n_sel)))  (Eq. 5).

    Reading of the ceiling: rho arrives as a double; when rho*n_sel lies within
    1e-9*max(1, n_sel) of an integer, that integer is taken (so 14% of 2,250 is
    315, as intended, not 316 from the binary representation of 0.14); otherwise
    the ceiling of the double product.  n_sel = 0 gives k = 0."""
    if not (0.0 <= rho <= 1.0) or math.isnan(rho):
        raise ValueError("density must lie in [0, 1]")
    p = float(rho) * float(n_sel)
    r = round(p)
    c = r if abs(p - r) <= 1e-9 * max(1, n_sel) else math.ceil(p)
    return min(n_sel, max(1, c))


# --------------------------------------------------------------------------
# Eq. (2): aggregated query-key block score
# --------------------------------------------------------------------------
def block_scores(q_bar: np.ndarray, k_bar: np.ndarray, d: int, sel: list[int]) -> np.ndarray:
    """S_ij = tau * q_bar_i . k_bar_j with tau = D^-1/2  (Eq. 2), for j in J_sel.

    Returns [n_q, n_k] with NaN in the keep columns: keep blocks are never
    scored (Section 5.2)."""
    tau = 1.0 / math.sqrt(d)
    s = np.full((q_bar.shape[0], k_bar.shape[0]), np.nan, dtype=np.float64)
    if sel:
        s[:, sel] = tau * (q_bar @ k_bar[sel].T)
    return s


# --------------------------------------------------------------------------
# Eq. (6): retained support
# --------------------------------------------------------------------------
def topk_idx(scores_row: np.ndarray, sel: list[int], k: int) -> list[int]:
    """TopKIdx over J_sel of one score row: the k selectable blocks with the
    highest scores.  Tie rule (the paper is silent): among equal scores the lower
    block index wins."""
    order = sorted(sel, key=lambda j: (-scores_row[j], j))
    return order[:k]


def retained_support(scores_row: np.ndarray, keep_set: list[int], sel: list[int], k: int) -> list[int]:
    """A_i = J_keep  union  TopKIdx_{j in J_sel}(S_ij, k)  (Eq. 6), as an
    ascending list (the forward-only kv_indices row of Section 5.3)."""
    return sorted(set(keep_set) | set(topk_idx(scores_row, sel, k)))


def select(q: np.ndarray, k: np.ndarray, b: int, rho: float, keep: list[tuple[int, int]]):
    """The whole selector for one head (Sections 5.1-5.2): pool, score, keep,
    budget, top-k.  Returns (lists, scores, k_budget, keep_set) where lists[i]
    is the ascending A_i of query block i."""
    lq, d = q.shape
    lk = k.shape[0]
    q_bar = pool(q, b)
    k_bar = pool(k, b)
    keep_set = keep_blocks(keep, lk, b)
    sel = selectable_blocks(keep_set, lk, b)
    kk = budget_k(rho, len(sel))
    s = block_scores(q_bar, k_bar, d, sel)
    lists = [retained_support(s[i], keep_set, sel, kk) for i in range(num_blocks(lq, b))]
    return lists, s, kk, keep_set


# --------------------------------------------------------------------------
# Eq. (7): block-sparse attention forward
# --------------------------------------------------------------------------
def sparse_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, lists: list[list[int]], b: int,
                     scale: float | None = None):
    """Forward attention under the token mask M_tu = 1[pi_k(u) in A_{pi_q(t)}] (Eq. 7).

    For each query token t of block i the visible keys are the tokens u < L_k of
    the blocks in A_i (padding positions of a partial final key block are masked,
    Section 5.3).  logits z = scale * q_t . k_u (scale defaults to D^-1/2),
    O_t = sum_u softmax(z)_u v_u and lse_t = ln sum_u exp(z_u).  A row with no
    visible key gets O = 0 and lse = -inf.  Returns (O [L_q, D], lse [L_q])."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    lq, d = q.shape
    lk = k.shape[0]
    s = (1.0 / math.sqrt(d)) if scale is None else float(scale)
    out = np.zeros((lq, v.shape[1]), dtype=np.float64)
    lse = np.full(lq, -np.inf, dtype=np.float64)
    for i in range(num_blocks(lq, b)):
        t0, t1 = block_token_range(i, lq, b)
        cols = [u for j in lists[i] for u in range(*block_token_range(j, lk, b))]
        if not cols:
            continue
        z = s * (q[t0:t1] @ k[cols].T)                # [rows, |U_i|]
        m = z.max(axis=1, keepdims=True)
        p = np.exp(z - m)
        l = p.sum(axis=1, keepdims=True)
        out[t0:t1] = (p @ v[cols]) / l
        lse[t0:t1] = (m + np.log(l))[:, 0]
    return out, lse


def dense_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float | None = None):
    """Plain softmax attention of every query over every key: the dense
    comparison (FlashAttention-2's role in Section 6), with no blocks at all."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    s = (1.0 / math.sqrt(q.shape[1])) if scale is None else float(scale)
    z = s * (q @ k.T)
    m = z.max(axis=1, keepdims=True)
    p = np.exp(z - m)
    l = p.sum(axis=1, keepdims=True)
    return (p @ v) / l, (m + np.log(l))[:, 0]


def token_mask(lists: list[list[int]], lq: int, lk: int, b: int) -> np.ndarray:
    """The boolean [L_q, L_k] token mask M of Eq. (7) (True = attend)."""
    m = np.zeros((lq, lk), dtype=bool)
    for i in range(num_blocks(lq, b)):
        t0, t1 = block_token_range(i, lq, b)
        for j in lists[i]:
            u0, u1 = block_token_range(j, lk, b)
            m[t0:t1, u0:u1] = True
    return m


# --------------------------------------------------------------------------
# Section 4 (Analysis): retained attention mass
# --------------------------------------------------------------------------
def _dense_probs(q: np.ndarray, k: np.ndarray, scale: float | None) -> np.ndarray:
    """Row-wise softmax of scale * Q K^T over every key (float64)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    s = (1.0 / math.sqrt(q.shape[1])) if scale is None else float(scale)
    z = s * (q @ k.T)
    p = np.exp(z - z.max(axis=1, keepdims=True))
    return p / p.sum(axis=1, keepdims=True)


def retained_mass(q: np.ndarray, k: np.ndarray, lists: list[list[int]], b: int,
                  scale: float | None = None) -> np.ndarray:
    """Share of each query's dense softmax mass that falls on the keys its block
    selection keeps: sum over u in the blocks of A_i (u < L_k) of
    softmax_u(scale * q_t . k_u), the retained attention mass the paper's
    analysis compares across selection strategies.  Returns [L_q]."""
    p = _dense_probs(q, k, scale)
    lq, lk = p.shape
    out = np.zeros(lq, dtype=np.float64)
    for i in range(num_blocks(lq, b)):
        t0, t1 = block_token_range(i, lq, b)
        cols = [u for j in lists[i] for u in range(*block_token_range(j, lk, b))]
        if cols:
            out[t0:t1] = p[t0:t1][:, cols].sum(axis=1)
    return out


def token_topk_mass(q: np.ndarray, k: np.ndarray, n_tokens: np.ndarray, scale: float | None = None) -> np.ndarray:
    """The token-wise upper bound: for each query t, the largest softmax mass
    any n_tokens[t] keys can hold, i.e. the sum of its n_tokens[t] largest
    dense softmax weights.  Returns [L_q]."""
    p = _dense_probs(q, k, scale)
    srt = -np.sort(-p, axis=1)
    n = np.asarray(n_tokens, dtype=np.int64)
    return np.array([srt[t, : max(0, min(int(n[t]), p.shape[1]))].sum() for t in range(p.shape[0])])

