"""fp64 reference of the SPLA decode step: test infrastructure only.

Only the test-suite, the smoke check and the CPU-baseline leg of the benchmark
may import this module. It is a plain, slow, step-by-step statement of what
the decode step computes, written from the paper (arXiv 2601.22379,
Sections 2.1-2.2 and 3.1-3.3) in float64 NumPy. It shares no code with the
HIP library.

Notation follows the paper: B block size, G query heads per KV head (GQA
group), k selected blocks, d head dimension, N (here L) cached tokens.
Query head m belongs to KV head floor(m / G) (contiguous groups, Sec. 2.2).

Readings taken where the paper leaves a detail open (each is repeated at the
step it affects):

* softmax scale s: Eq. (1) writes exp(q k^T) without a scale; the model uses
  the usual 1/sqrt(d) attention scale, which is applied to the exact logits
  and, because the block score estimates the same exp-mass, inside the
  Taylor estimate as well (s q in place of q). phi is applied to the
  unscaled vectors.
* phi is the softmax over the feature dimension (Sec. 3.2, "Numerical
  Stability"), max-shifted.
* the block covariance is the population (1/n) covariance of the block's
  keys, kept diagonal (Sec. 3.1); a partial last block uses its real count
  n_i in place of B.
* each head's block mass is normalised by that head's own Z over all blocks
  before the G heads are summed (Eq. 6 with Eq. 9).
* forced blocks (one sink block, the most recent n_local blocks; Sec. 4
  "Sparsity Specifications") count inside the budget k; the rest is top-k by
  score with ties going to the lower block index. If nb <= k every block is
  selected.
* the exact branch normalises over the selected tokens only (Eq. 5).
* the residual linear branch is unnormalised as written in Eqs. (15)-(16);
  when no token is left unselected the residual is exactly zero (decided by
  a count, not by a float test) and the output is the exact branch alone, so
  eps = 0 is allowed; an optional normaliser <phi(q), z_bar - z_sel> exists
  behind a flag.
* the combine adds an RMSNorm (per query head, over d, no mean subtraction,
  weight gamma, eps 1e-6) of the residual to the exact output, with no gate
  beyond gamma (Sec. 3.3).
* an empty sequence (L = 0) decodes to a zero output with no selection.
* prefill (Sec. 2 extends the decode formulation to prefill and training):
  the query at position t gets exactly the output a decode step at t would,
  over the first t + 1 tokens, including the statistics of its own partial
  block and S_bar over that prefix.
* strided block selection (Sec. 3.1, "Strided Block Selection"; optional):
  window w covers tokens [w s, min(w s + C, L)), one window per start below
  L, so the last windows may be partial and use their real counts. Each
  window gets the Taylor mass of its own keys; the per-head normaliser Z sums
  the masses of all windows; the group score of a window is Eq. (6) over
  windows; a block's relevance is the maximum group score over every window
  that shares a token with the block. With C = s = B the windows are the
  blocks and nothing changes.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional, Sequence

import numpy as np

f64 = np.float64


@dataclass(frozen=True)
class SplaParams:
    """Hyper-parameters of one SPLA attention layer at decode time.

    block_size (B), top_k (k), n_sink / n_local (forced blocks, Sec. 4
    "Sparsity Specifications": one sink block and the 4 most recent blocks),
    softmax_scale (None means 1/sqrt(d)), rms_eps (RMSNorm epsilon), and the
    ablation switches of Sec. 4 "Baselines": first_order (Eq. 11 instead of
    Eq. 10), no_rla (SPA: drop the residual linear branch), rla_normalize
    (divide the residual by its linear-attention normaliser).
    """

    block_size: int
    top_k: int
    n_sink: int = 1
    n_local: int = 4
    softmax_scale: Optional[float] = None
    rms_eps: float = 1e-6
    first_order: bool = False
    no_rla: bool = False
    rla_normalize: bool = False
    window: Optional[int] = None
    stride: Optional[int] = None

    def scale(self, d: int) -> float:
        return (1.0 / math.sqrt(d)) if self.softmax_scale is None else float(self.softmax_scale)

    def windows(self):
        """(C, s) of the selection windows; one window per block (C = s = B)
        unless window and stride are given (the paper's runs: C = 32, s = 16)."""
        C = self.block_size if self.window is None else int(self.window)
        st = self.block_size if self.stride is None else int(self.stride)
        if not 1 <= st <= C:
            raise ValueError("selection windows need 1 <= stride <= window")
        return C, st


@dataclass
class KVState:
    """What the append step maintains for one KV head (Sec. 3.1 and Eq. 15).

    mean, var: [n, d] key mean and diagonal population variance of each
    scoring unit; counts: [n] tokens per unit; s_bar: [d, d] global
    linear-attention state; z_bar: [d] sum of phi(k) (kept for the optional
    normaliser). The units are the blocks when window is None, else the
    selection windows of size window and stride stride.
    """

    mean: np.ndarray
    var: np.ndarray
    counts: np.ndarray
    s_bar: np.ndarray
    z_bar: np.ndarray
    length: int
    window: Optional[int] = None
    stride: Optional[int] = None


@dataclass
class DecodeResult:
    """Everything the decode step produces for one KV head group.

    out [G, d]; sel: selected block ids ascending (length <= k); score [nb];
    ell [G, n] per-head log mass of the n scoring units (the blocks, or the
    selection windows, whose group scores are then extras["window_score"]);
    o_sparse [G, d]; r [G, d] residual (zero when nothing is unselected or
    the RLA branch is off); o_bar and o_tilde [G, d]; n_forced: number of
    forced blocks (0 when nb <= k).
    """

    out: np.ndarray
    sel: np.ndarray
    score: np.ndarray
    ell: np.ndarray
    o_sparse: np.ndarray
    r: np.ndarray
    o_bar: np.ndarray
    o_tilde: np.ndarray
    n_forced: int
    extras: dict = field(default_factory=dict)


# ---------------------------------------------------------------- O1 blocks
def block_ranges(L: int, B: int) -> list:
    """Token ranges of the blocks (Sec. 2.1, Eq. 2: k_[i] = k_{(i-1)B+1 : iB}).

    0-based: block i holds tokens [iB, min((i+1)B, L)); nb = ceil(L / B).
    The last block may be partial.
    """
    nb = -(-L // B)
    return [(i * B, min((i + 1) * B, L)) for i in range(nb)]


# ----------------------------------------------------------------- O2 stats
def block_stats(K: np.ndarray, L: int, B: int):
    """Per-block key mean and diagonal covariance (Sec. 3.1).

    The second-order estimate, Eq. (10), needs the block mean k_bar and
    Cov(k); the paper keeps only the diagonal of Cov. Reading: population
    covariance (the estimate is an expectation over the block's own tokens),
    so a one-token block has zero variance.
    Returns mean [nb, d], var [nb, d], counts [nb].
    """
    K = np.asarray(K, dtype=f64)
    ranges = block_ranges(L, B)
    d = K.shape[-1]
    mean = np.zeros((len(ranges), d), dtype=f64)
    var = np.zeros((len(ranges), d), dtype=f64)
    counts = np.zeros(len(ranges), dtype=np.int64)
    for i, (a, b) in enumerate(ranges):
        blk = K[a:b]
        mean[i] = blk.mean(axis=0)
        var[i] = ((blk - mean[i]) ** 2).mean(axis=0)
        counts[i] = b - a
    return mean, var, counts


def window_ranges(L: int, C: int, s: int) -> list:
    """Token ranges of the strided selection windows (Sec. 3.1, "Strided
    Block Selection": windows of C tokens every s tokens). 0-based: window w
    holds tokens [ws, min(ws + C, L)) for every start ws < L, so the last
    windows may be partial."""
    nw = -(-L // s)
    return [(w * s, min(w * s + C, L)) for w in range(nw)]


def window_stats(K: np.ndarray, L: int, C: int, s: int):
    """Key mean and diagonal population covariance of every selection window
    (the block statistics of Sec. 3.1 taken over a window's tokens).
    Returns mean [nw, d], var [nw, d], counts [nw]."""
    K = np.asarray(K, dtype=f64)
    ranges = window_ranges(L, C, s)
    d = K.shape[-1]
    mean = np.zeros((len(ranges), d), dtype=f64)
    var = np.zeros((len(ranges), d), dtype=f64)
    counts = np.zeros(len(ranges), dtype=np.int64)
    for w, (a, b) in enumerate(ranges):
        win = K[a:b]
        mean[w] = win.mean(axis=0)
        var[w] = ((win - mean[w]) ** 2).mean(axis=0)
        counts[w] = b - a
    return mean, var, counts


def pool_windows_to_blocks(wscore: np.ndarray, L: int, B: int, C: int, s: int) -> np.ndarray:
    """Block relevance by max-pooling window scores (Sec. 3.1, "Strided
    Block Selection"). Reading: block i takes the largest score among the
    windows that share at least one token with it. Returns score [nb]."""
    wscore = np.asarray(wscore, dtype=f64)
    wr = np.array(window_ranges(L, C, s), dtype=np.int64).reshape(-1, 2)
    out = np.zeros(-(-L // B), dtype=f64)
    for i, (a, b) in enumerate(block_ranges(L, B)):
        touching = (wr[:, 0] < b) & (wr[:, 1] > a)
        out[i] = wscore[touching].max()
    return out


# ---------------------------------------------------------- O3 feature map
def feature_map(x: np.ndarray) -> np.ndarray:
    """phi(x) = softmax(x) over the feature dimension (Sec. 3.2, "Numerical
    Stability"; the exponential map phi(x) ~ exp(x) of "Parameterization",
    normalised). Applied to the unscaled query / key vectors."""
    x = np.asarray(x, dtype=f64)
    e = np.exp(x - x.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


# --------------------------------------------------------- O4 global state
def global_state(K: np.ndarray, V: np.ndarray, L: int):
    """Global linear-attention state after L tokens, Eq. (15):
    S_bar = sum_t phi(k_t)^T v_t  ([d, d]); also z_bar = sum_t phi(k_t)."""
    K = np.asarray(K, dtype=f64)[:L]
    V = np.asarray(V, dtype=f64)[:L]
    phik = feature_map(K)
    return phik.T @ V, phik.sum(axis=0)


# ------------------------------------------------------------ O5 log mass
def log_block_mass(q: np.ndarray, mean: np.ndarray, var: np.ndarray, counts: np.ndarray,
                   s: float, first_order: bool = False) -> np.ndarray:
    """Log of the estimated block mass, per head (Eqs. 8 and 10, Sec. 3.1).

    The mass of block i for head m is sum_{j in block} exp(s q_m . k_j)
    = n_i * E_j[exp(s q_m . k_j)] (Eq. 8, with the real count n_i). The
    expectation is replaced by the second-order Taylor estimate around the
    block mean, Eq. (10), exp(s q.mu)(1 + 1/2 (s q)^T Cov (s q)), with the
    diagonal covariance, so
        ell_m(i) = s q_m.mu_i + ln n_i + ln(1 + 1/2 s^2 sum_j q_mj^2 var_ij).
    first_order uses Eq. (11) and drops the last term.
    Returns ell [G, nb].
    """
    q = np.asarray(q, dtype=f64)
    ell = s * (q @ mean.T) + np.log(counts.astype(f64))[None, :]
    if not first_order:
        ell = ell + np.log1p(0.5 * s * s * ((q * q) @ var.T))
    return ell


# ---------------------------------------------------------- O6 group score
def group_block_scores(ell: np.ndarray) -> np.ndarray:
    """Group block score, Eq. (6): sum over the G heads of each head's block
    mass divided by that head's normaliser Z (Eq. 9, the sum of the masses of
    all blocks). Done in log space: p_m(i) = exp(ell_m(i) - LSE_i ell_m).
    Returns score [nb]; each head contributes a distribution over blocks,
    so the scores sum to G."""
    ell = np.asarray(ell, dtype=f64)
    mx = ell.max(axis=1, keepdims=True)
    lse = mx + np.log(np.exp(ell - mx).sum(axis=1, keepdims=True))
    return np.exp(ell - lse).sum(axis=0)


# ------------------------------------------------------------- O7 select
def forced_blocks(nb: int, k: int, n_sink: int, n_local: int) -> list:
    """Blocks always selected (Sec. 4, "Sparsity Specifications"): the first
    n_sink blocks (attention sink) and the n_local most recent blocks. None
    when nb <= k (then every block is selected anyway)."""
    if nb <= k:
        return []
    return sorted(set(range(min(n_sink, nb))) | set(range(max(nb - n_local, 0), nb)))


def select_blocks(score: np.ndarray, k: int, n_sink: int, n_local: int) -> np.ndarray:
    """Select operator of Eq. (3) with Select = TopK (Sec. 2.1).

    nb <= k: every block. Otherwise the forced blocks plus the top
    (k - |forced|) of the remaining blocks by score, descending; equal
    scores go to the lower block index. Forced blocks count inside k.
    Returns the selected block ids in ascending order.
    """
    nb = len(score)
    if nb <= k:
        return np.arange(nb, dtype=np.int64)
    forced = forced_blocks(nb, k, n_sink, n_local)
    fset = set(forced)
    rest = [i for i in range(nb) if i not in fset]
    rest.sort(key=lambda i: (-float(score[i]), i))
    chosen = forced + rest[: k - len(forced)]
    return np.array(sorted(chosen), dtype=np.int64)


def cutoff_score(score: np.ndarray, sel: np.ndarray, k: int, n_sink: int, n_local: int):
    """Score of the last block admitted by rank (the lowest-scored non-forced
    selected block), or None when every block is selected."""
    nb = len(score)
    if nb <= k:
        return None
    fset = set(forced_blocks(nb, k, n_sink, n_local))
    ranked = [float(score[i]) for i in sel if int(i) not in fset]
    return min(ranked) if ranked else None


def selected_token_indices(sel: Sequence[int], L: int, B: int) -> np.ndarray:
    """Tokens of the selected blocks (the set T_I of Eq. 2), ascending."""
    parts = [np.arange(i * B, min((i + 1) * B, L)) for i in sel]
    return np.concatenate(parts) if parts else np.zeros(0, dtype=np.int64)


# ----------------------------------------------------------- O8 exact
def exact_sparse_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray, tok: np.ndarray,
                           s: float) -> np.ndarray:
    """Grouped block-sparse attention, Eq. (5): softmax attention of the G
    query heads over the selected tokens only; Z runs row-wise over the
    selected tokens. Returns o_sparse [G, d]."""
    q = np.asarray(q, dtype=f64)
    if len(tok) == 0:
        return np.zeros_like(q)
    Ks = np.asarray(K, dtype=f64)[tok]
    Vs = np.asarray(V, dtype=f64)[tok]
    a = s * (q @ Ks.T)
    a = a - a.max(axis=1, keepdims=True)
    p = np.exp(a)
    p = p / p.sum(axis=1, keepdims=True)
    return p @ Vs


# ------------------------------------------------------------- O9 RLA
def nothing_unselected(n_selected_tokens: int, L: int) -> bool:
    """Whether the selection holds every cached token, so the residual
    branch of Eq. (14) has no token to cover. Decided by a count, never by
    testing a float for zero."""
    return int(n_selected_tokens) == int(L)


def residual_linear_attention(q: np.ndarray, s_bar: np.ndarray, z_bar: np.ndarray,
                              K: np.ndarray, V: np.ndarray, tok: np.ndarray, L: int,
                              normalize: bool = False):
    """Residual linear attention by subtraction, Eqs. (14)-(16).

    o_bar = phi(q) S_bar (Eq. 15), o_tilde = phi(q) S_tilde with S_tilde
    summed over the selected tokens only (Eq. 16), r = o_bar - o_tilde
    (Eq. 14). When every token is selected r is exactly 0. With normalize,
    r is divided by <phi(q), z_bar - z_tilde>.
    Returns (r, o_bar, o_tilde), each [G, d].
    """
    phiq = feature_map(q)
    o_bar = phiq @ s_bar
    if len(tok) > 0:
        phik = feature_map(np.asarray(K, dtype=f64)[tok])
        o_tilde = (phiq @ phik.T) @ np.asarray(V, dtype=f64)[tok]
        z_tilde = phik.sum(axis=0)
    else:
        o_tilde = np.zeros_like(o_bar)
        z_tilde = np.zeros_like(z_bar)
    if nothing_unselected(len(tok), L):
        return np.zeros_like(o_bar), o_bar, o_tilde
    r = o_bar - o_tilde
    if normalize:
        r = r / (phiq @ (z_bar - z_tilde))[:, None]
    return r, o_bar, o_tilde


# ------------------------------------------------------------ O10 combine
def combine(o_sparse: np.ndarray, r: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """SPLA output (Sec. 3.3): o = o_sparse + RMSNorm(o_rla), the RMSNorm per
    query head over d with weight gamma and epsilon eps."""
    r = np.asarray(r, dtype=f64)
    rms = np.sqrt((r * r).mean(axis=-1, keepdims=True) + eps)
    return o_sparse + np.asarray(gamma, dtype=f64) * r / rms


# ------------------------------------------------------ state and decode
def build_state(K: np.ndarray, V: np.ndarray, L: int, B: int,
                window: Optional[int] = None, stride: Optional[int] = None) -> KVState:
    """State of one KV head after its first L tokens were appended; the
    statistics are per block, or per selection window when window and
    stride are given (C = s = B is the block path)."""
    if (window, stride) == (B, B):
        window = stride = None
    if window is None and stride is None:
        mean, var, counts = block_stats(K, L, B)
    else:
        mean, var, counts = window_stats(K, L, window, stride)
    s_bar, z_bar = global_state(K, V, L)
    return KVState(mean, var, counts, s_bar, z_bar, L, window, stride)


def append_state(state: Optional[KVState], k_new: np.ndarray, v_new: np.ndarray, B: int,
                 d: Optional[int] = None, window: Optional[int] = None,
                 stride: Optional[int] = None) -> KVState:
    """Streaming append of tokens, one at a time (Eq. 15 for the state; the
    statistics of every unit that holds the token updated with Welford's
    recurrence for the mean and the sum of squared deviations). The units are
    the blocks, or the selection windows when window and stride are given: a
    token at position t lies in the windows whose start ws satisfies
    ws <= t < ws + C. A decode issued after an append sees the appended tokens
    (the query at position N attends to 1..N, Sec. 2)."""
    k_new = np.asarray(k_new, dtype=f64)
    v_new = np.asarray(v_new, dtype=f64)
    if (window, stride) == (B, B):
        window = stride = None
    if d is None:
        d = k_new.shape[-1]
    if state is None:
        state = KVState(np.zeros((0, d)), np.zeros((0, d)), np.zeros(0, dtype=np.int64),
                        np.zeros((d, d)), np.zeros(d), 0, window, stride)
    elif (state.window, state.stride) != (window, stride):
        raise ValueError("append with other selection windows than the state holds")
    C = B if window is None else window
    st = B if stride is None else stride
    mean = [row.copy() for row in state.mean]
    m2 = [state.var[i] * state.counts[i] for i in range(len(state.counts))]
    counts = [int(c) for c in state.counts]
    s_bar = state.s_bar.copy()
    z_bar = state.z_bar.copy()
    L = state.length
    for k, v in zip(k_new, v_new):
        if L % st == 0:  # token L opens unit L / s
            mean.append(np.zeros(d))
            m2.append(np.zeros(d))
            counts.append(0)
        for i in range(max(0, len(counts) - C // st - 2), len(counts)):
            if not i * st <= L < i * st + C:
                continue
            counts[i] += 1
            delta = k - mean[i]
            mean[i] = mean[i] + delta / counts[i]
            m2[i] = m2[i] + delta * (k - mean[i])
        phik = feature_map(k)
        s_bar += np.outer(phik, v)
        z_bar += phik
        L += 1
    cnt = np.array(counts, dtype=np.int64)
    var = np.array([m2[i] / counts[i] for i in range(len(counts))]).reshape(-1, d)
    return KVState(np.array(mean).reshape(-1, d), var, cnt, s_bar, z_bar, L, window, stride)


def decode_kv_head(q: np.ndarray, state: KVState, K: np.ndarray, V: np.ndarray,
                   gamma: np.ndarray, p: SplaParams,
                   force_selection: Optional[Sequence[int]] = None) -> DecodeResult:
    """Decode step for the G query heads of one KV head (Secs. 2.2, 3.1-3.3).

    q [G, d]; state built from the first state.length rows of K, V [>=L, d];
    gamma [G, d]. force_selection replaces the selected block set (used to
    compare outputs when two correct selections differ by a near tie).
    """
    q = np.asarray(q, dtype=f64)
    G, d = q.shape
    L = state.length
    B, k = p.block_size, p.top_k
    if L == 0:
        z = np.zeros((G, d))
        return DecodeResult(z.copy(), np.zeros(0, dtype=np.int64), np.zeros(0), np.zeros((G, 0)),
                            z.copy(), z.copy(), z.copy(), z.copy(), 0)
    s = p.scale(d)
    C, st = p.windows()
    strided = (C, st) != (B, B)
    if (state.window, state.stride) != ((C, st) if strided else (None, None)):
        raise ValueError("the state's statistics are not over the selection windows of p")
    # per-unit (block, or window) log mass and Eq. (6) group score over units
    ell = log_block_mass(q, state.mean, state.var, state.counts, s, p.first_order)
    score = group_block_scores(ell)
    extras = {}
    if strided:
        extras["window_score"] = score
        score = pool_windows_to_blocks(score, L, B, C, st)
    nb = len(score)
    if force_selection is None:
        sel = select_blocks(score, k, p.n_sink, p.n_local)
    else:
        sel = np.array(sorted(int(i) for i in force_selection), dtype=np.int64)
    n_forced = len(forced_blocks(nb, k, p.n_sink, p.n_local))
    tok = selected_token_indices(sel, L, B)
    o_sparse = exact_sparse_attention(q, K, V, tok, s)
    if p.no_rla:
        z = np.zeros_like(o_sparse)
        return DecodeResult(o_sparse.copy(), sel, score, ell, o_sparse, z, z.copy(), z.copy(),
                            n_forced, extras)
    r, o_bar, o_tilde = residual_linear_attention(q, state.s_bar, state.z_bar, K, V, tok, L,
                                                  p.rla_normalize)
    if nothing_unselected(len(tok), L):
        # no unselected token: the residual branch is absent, so its RMSNorm
        # term is zero (also at eps = 0, where gamma 0 / sqrt(0) is undefined)
        out = o_sparse.copy()
    else:
        out = combine(o_sparse, r, gamma, p.rms_eps)
    return DecodeResult(out, sel, score, ell, o_sparse, r, o_bar, o_tilde, n_forced, extras)


def decode_from_state(q: np.ndarray, states: Sequence[KVState], K: np.ndarray, V: np.ndarray,
                      gamma: np.ndarray, p: SplaParams, force_selection=None):
    """Decode step of one sequence. q [Hq, d]; states one per KV head;
    K, V [Hkv, >=L, d]; gamma [Hq, d]. force_selection: None or a list of
    per-KV-head block id lists. Returns a list of DecodeResult, one per KV
    head (query heads h*G .. h*G+G-1)."""
    q = np.asarray(q, dtype=f64)
    Hq = q.shape[0]
    Hkv = len(states)
    G = Hq // Hkv
    out = []
    for h in range(Hkv):
        fs = None if force_selection is None else force_selection[h]
        out.append(decode_kv_head(q[h * G:(h + 1) * G], states[h], K[h], V[h],
                                  gamma[h * G:(h + 1) * G], p, fs))
    return out


def decode_sequence(q: np.ndarray, K: np.ndarray, V: np.ndarray, L: int, gamma: np.ndarray,
                    p: SplaParams, force_selection=None):
    """Append the first L tokens of every KV head, then decode q."""
    C, st = p.windows()
    win = (None, None) if (C, st) == (p.block_size, p.block_size) else (C, st)
    states = [build_state(K[h], V[h], L, p.block_size, *win) for h in range(K.shape[0])]
    return decode_from_state(q, states, K, V, gamma, p, force_selection)


# ------------------------------------------------------- chunked prefill
def prefill_kv_head(Q: np.ndarray, K: np.ndarray, V: np.ndarray, L0: int, gamma: np.ndarray,
                    p: SplaParams) -> list:
    """Causal prefill of one KV head group (Sec. 2: the decode formulation
    carries over to prefill and training). Q [T, G, d] are the queries at
    positions L0 .. L0 + T - 1; K, V [>= L0 + T, d]. The query at position t
    sees the tokens 0 .. t, so its output is the decode step on the state of
    the first t + 1 tokens: its own block selection (the block holding t is
    partial and its statistics cover tokens up to t), the exact branch over
    the selected tokens, and the residual linear branch with S_bar taken over
    the same prefix. Returns a list of T DecodeResult."""
    Q = np.asarray(Q, dtype=f64)
    C, st = p.windows()
    win = (None, None) if (C, st) == (p.block_size, p.block_size) else (C, st)
    out = []
    for i in range(Q.shape[0]):
        n = L0 + i + 1
        state = build_state(K, V, n, p.block_size, *win)
        out.append(decode_kv_head(Q[i], state, K[:n], V[:n], gamma, p))
    return out
