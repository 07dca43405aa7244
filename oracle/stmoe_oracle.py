"""Plain CPU oracle for the ST-MoE decode-step MoE layer.

TEST INFRASTRUCTURE.  Only the test suite, the package smoke check and the
benchmark's CPU-baseline leg may import or call this module.  The product path
never does, and this module imports nothing from the product package: it takes
the seeded input arrays as arguments and shares no code with the HIP path.

Arithmetic: float64 for every floating-point step, integer numpy arrays for
the prediction tables.  Each function names the passage of the paper it
follows and states it in its own terms (set and membership-matrix form), not
as a transcription of the printed listings.

Parity status per function (see the pins under ``tests/``):
  router_logits / softmax_rows / topk_rows / route   pinned (invariants, brute force)
  swiglu_expert / moe_ffn                            pinned (explicit triple loop, special cases)
  STPredictor.profile / update / predict             pinned (hand-worked example, invariants,
                                                      closed form K^2/N, special cases,
                                                      exhaustive update check on E = 4)
  CacheSim, admitted, warm_from_profile, use_counts  pinned (hand-worked traces, invariants,
                                                      exhaustive optimum lower bound; the
                                                      frequency-aware rule by a hand trace)
  decode_reference (the per-layer loop)              pinned (hand-worked five-token run:
                                                      per-token hits, scores, tables, the
                                                      capped cache's copy log in both modes,
                                                      frozen tables; planted slips fail it).
                                                      Its hit rates and stall on synthetic
                                                      inputs have no paper value: those
                                                      absolute numbers are parity unpinned
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

NEAR_TIE = 1e-4      # routing decisions closer than this are exempt from exact parity
CONF_INIT = 2        # 2-bit state "10": preferred (Alg. 1; HT entries, Section 4.2)
CONF_MAX = 3         # 2-bit state "11": strongly preferred (Alg. 3)
THRESHOLD = 2        # prefetch threshold, state "10" (Alg. 2, text after it)
HT_SCORE = 2         # HT confidences are fixed at "10" (Section 4.2, History Table)


# ----------------------------------------------------------------------------
# format decoding (the oracle's own copy; the HIP side decodes in its kernels)
# ----------------------------------------------------------------------------

def decode_storage(a: np.ndarray) -> np.ndarray:
    """Storage array (uint16 bfloat16 bit patterns or float32) -> exact float64 values."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


# ----------------------------------------------------------------------------
# gating (Section 2: z_j = w_j^T x, softmax, top-K, probability-weighted sum)
# ----------------------------------------------------------------------------

def router_logits(x: np.ndarray, wg: np.ndarray) -> np.ndarray:
    """z[b][e] = w_e^T x_b in float64 (Section 2)."""
    return np.asarray(x, np.float64) @ np.asarray(wg, np.float64).T


def softmax_rows(z: np.ndarray) -> np.ndarray:
    """s = softmax(z) per row, max-subtracted (Section 2)."""
    m = z.max(axis=1, keepdims=True)
    e = np.exp(z - m)
    return e / e.sum(axis=1, keepdims=True)


def topk_rows(z: np.ndarray, K: int) -> np.ndarray:
    """Top-K experts per row by logit, descending; equal logits -> lower index first.

    Softmax is monotone, so the top-K gating probabilities (Section 2) are the
    top-K logits; comparing logits avoids ties created by rounding probabilities.
    """
    out = np.empty((z.shape[0], K), dtype=np.int64)
    for b in range(z.shape[0]):
        order = sorted(range(z.shape[1]), key=lambda e: (-z[b, e], e))
        out[b] = order[:K]
    return out


def near_ties(z: np.ndarray, K: int, eps: float = NEAR_TIE):
    """Per row: (boundary, order) flags.

    boundary: the K-th and (K+1)-th largest logits differ by less than eps, so
              the selected *set* may legitimately differ between precisions;
    order:    two adjacent logits among the top K differ by less than eps, so
              only their order within the selection may differ.
    """
    zs = -np.sort(-z, axis=1)
    E = z.shape[1]
    boundary = np.zeros(z.shape[0], bool)
    if K < E:
        boundary = (zs[:, K - 1] - zs[:, K]) < eps
    order = np.zeros(z.shape[0], bool)
    if K > 1:
        order = (np.diff(-zs[:, :K], axis=1) < eps).any(axis=1)
    return boundary, order


def route(x: np.ndarray, wg: np.ndarray, K: int, renorm: bool = False) -> dict:
    """Gating of Section 2 for a batch of tokens.

    Gate weights are the full-softmax probabilities of the selected experts
    (the paper weights outputs by their gating probabilities); ``renorm``
    divides them by their sum instead.
    """
    z = router_logits(x, wg)
    s = softmax_rows(z)
    idx = topk_rows(z, K)
    w = np.take_along_axis(s, idx, axis=1)
    if renorm:
        w = w / w.sum(axis=1, keepdims=True)
    boundary, order = near_ties(z, K)
    return dict(z=z, s=s, idx=idx, w=w, tie_boundary=boundary, tie_order=order)


# ----------------------------------------------------------------------------
# expert FFN (Section 2: experts are feed-forward networks; SwiGLU form)
# ----------------------------------------------------------------------------

def silu(g):
    return g / (1.0 + np.exp(-g))


def swiglu_expert(x: np.ndarray, w_gate: np.ndarray, w_up: np.ndarray, w_down: np.ndarray):
    """y = W_down (silu(W_gate x) * (W_up x)); x [..., H], W_gate/W_up [I][H], W_down [H][I]."""
    x = np.asarray(x, np.float64)
    g = x @ np.asarray(w_gate, np.float64).T
    u = x @ np.asarray(w_up, np.float64).T
    return (silu(g) * u) @ np.asarray(w_down, np.float64).T


def moe_ffn(x: np.ndarray, idx: np.ndarray, w: np.ndarray, expert, shared=()):
    """y[b] = sum_k w[b][k] * FFN_{idx[b][k]}(x[b]) + sum_s FFN_s(x[b]) (Section 2).

    ``expert(e)`` returns (W_gate, W_up, W_down) as float64; ``shared`` is a
    sequence of such triples for always-on experts (weight 1).
    """
    x = np.asarray(x, np.float64)
    y = np.zeros_like(x)
    cache = {}
    for b in range(x.shape[0]):
        for k in range(idx.shape[1]):
            e = int(idx[b, k])
            if e not in cache:
                cache[e] = expert(e)
            y[b] += w[b, k] * swiglu_expert(x[b], *cache[e])
        for mats in shared:
            y[b] += swiglu_expert(x[b], *mats)
    return y


# ----------------------------------------------------------------------------
# the spatio-temporal predictor (Section 4.2, Algorithms 1-3, Eq. 1)
# ----------------------------------------------------------------------------

class STPredictor:
    """Cross-layer Correlation Tables (one per adjacent layer pair) and a
    per-layer, per-batch-row History Table (Section 4.2).

    cct_idx[i][e][s], cct_conf[i][e][s]  (int64 arrays [L-1][E][K]): slot s of
        the CCT entry of expert e for the layer pair (i, i+1);
    ht[l][b]  (int64 array [L][B][K]): the previous token's selection at layer
        l for batch row b, sorted ascending (it is a set; its confidence is
        fixed at 2);
    co[i]  (int64 array [L-1][E][E]): the profiling co-activation counts.
    """

    def __init__(self, L: int, E: int, K: int, B: int = 1):
        self.L, self.E, self.K, self.B = L, E, K, B
        self.co = np.zeros((max(L - 1, 0), E, E), np.int64)
        self.cct_idx = np.zeros((max(L - 1, 0), E, K), np.int64)
        self.cct_conf = np.zeros((max(L - 1, 0), E, K), np.int64)
        self.ht = np.zeros((L, B, K), np.int64)

    def _indicator(self, sets) -> np.ndarray:
        """Rows of 0/1 membership vectors over the E experts."""
        sets = np.asarray(sets, np.int64).reshape(-1, self.K)
        m = np.zeros((sets.shape[0], self.E), np.int64)
        np.put_along_axis(m, sets, 1, axis=1)
        return m

    def profile(self, sel) -> None:
        """Build the tables from the profiling tokens (Algorithm 1; HT from
        Section 4.1 and the framework figure).

        sel[p][b][l][k]: the profiling tokens' selections.  With X_l the
        matrix of membership vectors of layer l's selections (one row per
        (token, batch row)), the co-activation counts of the pair (i, i+1) are
        X_i^T X_{i+1}: entry (e, f) counts the rows that chose e at layer i
        and f at layer i+1.  The CCT entry of e keeps the K experts with the
        largest counts (equal counts: lower index first, which also fixes the
        choice among all-zero tails), each with confidence 2.  The HT holds
        the last profiling token's selections.
        """
        sel = np.asarray(sel, np.int64)
        P = sel.shape[0]
        X = [self._indicator(sel[:, :, l, :]) for l in range(self.L)]
        for i in range(self.L - 1):
            self.co[i] = X[i].T @ X[i + 1]
            for e in range(self.E):
                # a stable sort on the negated counts keeps index order on ties
                self.cct_idx[i, e] = np.argsort(-self.co[i, e], kind="stable")[:self.K]
            self.cct_conf[i] = CONF_INIT
        self.ht[:] = np.sort(sel[P - 1].transpose(1, 0, 2), axis=2)

    def load_tables(self, cct_idx, cct_conf, ht) -> None:
        """Replace the CCTs and the HT (e.g. with planted wrong predictions)."""
        self.cct_idx[:] = np.asarray(cct_idx, np.int64)
        self.cct_conf[:] = np.asarray(cct_conf, np.int64)
        self.ht[:] = np.sort(np.asarray(ht, np.int64), axis=2)

    def update_entry(self, i: int, e: int, F) -> None:
        """Table update of one CCT entry against the actual next-layer set F
        (Algorithm 3; the CCT paragraph of Section 4.2).

        The entry's experts found in F are confirmed: their 2-bit confidence
        rises by one, saturating at 3.  Experts not in F lose one confidence
        level while they have one; those already at 0 make way for experts of
        F that the entry does not hold: the slots being replaced, taken in
        slot order, receive those experts in ascending order, with the initial
        confidence 2.  There are never more such slots than candidates (each
        unconfirmed slot leaves one expert of F unmatched), so the entry stays
        a set of K distinct experts.
        """
        row, conf = self.cct_idx[i, e], self.cct_conf[i, e]
        Fs = np.asarray(sorted(int(f) for f in F), np.int64)
        confirmed = np.isin(row, Fs)
        replaced = ~confirmed & (conf == 0)
        newcomers = np.setdiff1d(Fs, row)           # sorted, not held by the entry
        conf[:] = np.where(confirmed, np.minimum(conf + 1, CONF_MAX), conf - 1)
        row[replaced] = newcomers[:int(replaced.sum())]
        conf[replaced] = CONF_INIT

    def update(self, layer: int, prev_sets, cur_sets, online: bool = True) -> None:
        """Verify step at ``layer`` (Section 4.3.4, V): every CCT entry of the
        pair (layer-1, layer) that the previous layer selected is updated
        against this layer's selection (batch rows in order b = 0..B-1); then
        HT[layer][b] is overwritten with this token's selection.  online=False
        freezes the CCTs (the HT is still overwritten)."""
        if layer >= 1 and online:
            for b in range(self.B):
                for e in prev_sets[b]:
                    self.update_entry(layer - 1, int(e), cur_sets[b])
        for b in range(self.B):
            self.ht[layer, b] = sorted(int(v) for v in cur_sets[b])

    def predict(self, layer: int, cur_sets, use_cct: bool = True, use_ht: bool = True):
        """Eq. 1 scores of every expert for layer+1, per batch row.

        The spatial part sums, over the experts e selected at ``layer``, the
        confidence with which CCT[layer][e] names each candidate; the temporal
        part adds the fixed HT confidence 2 to the experts that the previous
        token selected at layer+1.  layer == -1 scores layer 0 from HT[0]
        alone (no earlier layer).  Returns an int64 array [B][E].
        """
        tgt = layer + 1
        sc = np.zeros((self.B, self.E), np.int64)
        for b in range(self.B):
            if use_cct and layer >= 0:
                A = np.asarray([int(e) for e in cur_sets[b]], np.int64)
                sc[b] += np.bincount(self.cct_idx[layer, A].ravel(),
                                     weights=self.cct_conf[layer, A].ravel(),
                                     minlength=self.E).astype(np.int64)
            if use_ht:
                sc[b, self.ht[tgt, b]] += HT_SCORE
        return sc

    @staticmethod
    def prefetch_sets(scores):
        """Per-row PrefetchSet: the experts whose score reaches the threshold 2
        (Algorithm 2 and the text after it)."""
        return [sorted(int(f) for f in np.nonzero(scores[b] >= THRESHOLD)[0])
                for b in range(scores.shape[0])]

    @staticmethod
    def ranked_union(scores):
        """Union of the rows' prefetch sets ranked by (max score desc, index asc)."""
        m = scores.max(axis=0)
        cand = [f for f in range(scores.shape[1]) if m[f] >= THRESHOLD]
        return sorted(cand, key=lambda f: (-int(m[f]), f))

    def tables(self):
        """Copies of (co [L-1][E][E], cct_idx [L-1][E][K], cct_conf [L-1][E][K], ht [L][B][K])."""
        return self.co.copy(), self.cct_idx.copy(), self.cct_conf.copy(), self.ht.copy()


# ----------------------------------------------------------------------------
# HBM expert cache policy (prefetch staging, Section 4.1 and 4.3.4)
# ----------------------------------------------------------------------------

@dataclass
class CacheCounts:
    hits: int = 0              # selected experts resident when demanded
    demand: int = 0            # demand ("missed loading") copies admitted to a slot
    overflow: int = 0          # demand copies streamed through staging (no free slot)
    prefetch: int = 0          # prefetch copies issued
    useful: int = 0            # prefetched experts that the layer then selected
    wasted: int = 0            # prefetched experts that the layer did not select
    log: list = field(default_factory=list)


class CacheSim:
    """Per-layer partition of C slots, least-recently-used with prediction protection.

    prefetch(l, ranked, stamp): for each ranked expert (at most C) that is not
    resident, evict the resident slot whose expert is not in the ranked set
    with the smallest (last_use, slot); stop when none is left.
    acquire(l, U, stamp): for each selected expert (ascending) that is not
    resident, evict the slot whose expert is not in U with the smallest
    (last_use, slot); with no such slot the copy streams through staging
    without admission.  Then every resident expert of U gets last_use = stamp.
    Residency counts from copy issue, so counts do not depend on timing.

    staged = n > 0 (an alternative use of the same prediction): prefetch copies
    the first n ranked experts that are not resident aside, changing no slot;
    acquire then decides exactly as without prefetching, except that a staged
    expert needs no copy (useful); staged experts not selected are wasted.

    counts [L][E] (frequency-aware eviction, an alternative replacement rule):
    the victim is the evictable slot with the smallest (use count of its
    expert, last_use, slot), an empty slot counting -1; every acquire adds 1
    to the count of each expert it is given.  counts=None: least recently
    used as above.
    """

    def __init__(self, L: int, E: int, C: int, warm=None, staged: int = 0, counts=None):
        self.L, self.E, self.C = L, E, C
        self.staged = staged
        self.freq = None if counts is None else [[int(v) for v in row] for row in counts]
        self.stage = [[] for _ in range(L)]
        self.slot = [[-1] * C for _ in range(L)]
        self.last = [[0] * C for _ in range(L)]
        self.pending = [set() for _ in range(L)]
        self.n = CacheCounts()
        if warm is not None:
            for l in range(L):
                for c in range(C):
                    self.slot[l][c] = int(warm[l][c])

    def _where(self, l, e):
        try:
            return self.slot[l].index(e)
        except ValueError:
            return -1

    def _victim(self, l, keep):
        cands = [c for c in range(self.C) if self.slot[l][c] not in keep]
        if not cands:
            return -1
        if self.freq is not None:
            def uses(c):
                e = self.slot[l][c]
                return self.freq[l][e] if e >= 0 else -1
            return min(cands, key=lambda c: (uses(c), self.last[l][c], c))
        return min(cands, key=lambda c: (self.last[l][c], c))

    def prefetch(self, l: int, ranked, stamp: int):
        if self.staged:
            # staged: the first `staged` ranked experts that are not resident are
            # copied aside; no slot changes hands
            copies = [f for f in (int(v) for v in ranked) if self._where(l, f) < 0][:self.staged]
            self.stage[l] = copies
            self.n.prefetch += len(copies)
            self.n.log.append(("P", l, stamp, tuple((f, -1) for f in copies)))
            return [(f, -1) for f in copies]
        ranked = [int(f) for f in ranked][:self.C]
        keep = set(ranked)
        copies = []
        for f in ranked:
            if self._where(l, f) >= 0:
                continue
            c = self._victim(l, keep)
            if c < 0:
                break
            self.slot[l][c] = f
            self.last[l][c] = stamp
            self.pending[l].add(f)
            copies.append((f, c))
        self.n.prefetch += len(copies)
        self.n.log.append(("P", l, stamp, tuple(copies)))
        return copies

    def acquire(self, l: int, U, stamp: int):
        U = sorted(set(int(f) for f in U))
        keep = set(U)
        where, demand, overflow = {}, [], []
        staged = set(self.stage[l])
        for f in U:
            c = self._where(l, f)
            if c >= 0:
                self.n.hits += 1
                where[f] = c
                continue
            c = self._victim(l, keep)
            if c < 0:
                if f not in staged:           # a staged expert is used from its staging copy
                    overflow.append(f)
                where[f] = -1
                continue
            self.slot[l][c] = f
            if f not in staged:               # a staged expert takes the slot without a copy
                demand.append((f, c))
            where[f] = c
        for f, c in where.items():
            if c >= 0:
                self.last[l][c] = stamp
        hits = sum(1 for f in U if f not in staged) - len(demand) - len(overflow)
        if self.staged:
            useful, wasted = len(staged & keep), len(staged - keep)
            self.stage[l] = []
        else:
            useful, wasted = len(self.pending[l] & keep), len(self.pending[l] - keep)
        self.n.demand += len(demand)
        self.n.overflow += len(overflow)
        self.n.useful += useful
        self.n.wasted += wasted
        self.pending[l] = set()
        if self.freq is not None:
            for f in U:
                self.freq[l][f] += 1
        self.n.log.append(("A", l, stamp, tuple(demand), tuple(overflow), hits, useful, wasted))
        return where, demand, overflow


# ----------------------------------------------------------------------------
# the per-layer decode loop (Section 4.3.4 workflow)
# ----------------------------------------------------------------------------

MODE_ON_DEMAND, MODE_STMOE, MODE_HT_ONLY, MODE_CCT_ONLY = 0, 1, 2, 3


def stamp_of(t: int, l: int, L: int) -> int:
    return t * L + l + 1


def admitted(scores, min_score: int = THRESHOLD, max_per_layer=None):
    """The prefix of the ranked union (max score desc, index asc) whose max
    score reaches ``min_score``, at most ``max_per_layer`` long: the experts a
    prefetch is issued for.  min_score = 2 with no cap is the paper's
    PrefetchSet (Algorithm 2); larger values are an admission ablation."""
    m = np.asarray(scores).max(axis=0)
    out = [f for f in STPredictor.ranked_union(scores) if m[f] >= min_score]
    return out if max_per_layer is None else out[:max_per_layer]


def warm_from_profile(prof_sel, L: int, E: int, C: int):
    """Initial cache residency: per layer, the C experts selected most often
    by the profiling tokens (count desc, index asc), -1 padding when C > E.
    sel[p][b][l][k] -> int64 [L][C]."""
    prof_sel = np.asarray(prof_sel, np.int64)
    out = np.full((L, C), -1, np.int64)
    for l in range(L):
        cnt = np.bincount(prof_sel[:, :, l, :].ravel(), minlength=E)
        order = sorted(range(E), key=lambda e: (-int(cnt[e]), e))[:min(C, E)]
        out[l, :len(order)] = order
    return out


def use_counts(prof_sel, L: int, E: int):
    """Seeds of frequency-aware eviction: per layer, the number of profiling
    tokens whose selection (any batch row) contains each expert.
    sel[p][b][l][k] -> int64 [L][E]."""
    prof_sel = np.asarray(prof_sel, np.int64)
    out = np.zeros((L, E), np.int64)
    for p in range(prof_sel.shape[0]):
        for l in range(L):
            out[l, np.unique(prof_sel[p, :, l, :])] += 1
    return out


def decode_reference(L, E, K, B, x_of, wg_of, prof_sel, n_tokens, C=None, warm=None,
                     mode=MODE_STMOE, renorm=False, ffn_of=None, ffn_tokens=0, online=True,
                     tables=None, min_score=THRESHOLD, max_per_layer=None, staged=0, counts=None):
    """Run the decode loop on the CPU.

    x_of(t, l) -> x [B][H] float64; wg_of(l) -> W_g [E][H] float64;
    ffn_of(l) -> callable(x, idx, w) -> y, used for the first ``ffn_tokens`` tokens.
    Per layer, in order: route; score this layer's prediction; Algorithm 3 on
    the previous layer pair and HT overwrite; predict the next layer (Eq. 1);
    demand-load the selection; FFN; prefetch the next layer's ranked set.
    online=False freezes the CCTs after profiling (Algorithm 3's confidence
    and replacement steps are skipped; HT is still overwritten).
    tables=(cct_idx, cct_conf, ht) replaces the profiled tables before the
    first token (planted wrong predictions).  min_score / max_per_layer are
    the prefetch admission knobs of ``admitted``; staged > 0 stages prefetches
    aside instead of evicting, counts switches the cache to frequency-aware
    eviction (CacheSim).
    Returns a dict of per-(t, l) records and totals.
    """
    pred = STPredictor(L, E, K, B)
    pred.profile(prof_sel)
    if tables is not None:
        pred.load_tables(*tables)
    use_cct = mode in (MODE_STMOE, MODE_CCT_ONLY)
    use_ht = mode in (MODE_STMOE, MODE_HT_ONLY)
    cache = CacheSim(L, E, C, warm, staged, counts) if C is not None else None
    # layer 0 of the first token is predicted from the profiled HT[0]
    P_cur = pred.predict(-1, None, use_cct=False, use_ht=use_ht)
    rec = dict(idx=[], w=[], scores=[], hits=np.zeros((n_tokens, L), np.int64),
               npred=np.zeros((n_tokens, L), np.int64), tie_boundary=0, tie_order=0, y={})
    if cache is not None and mode != MODE_ON_DEMAND:
        cache.prefetch(0, admitted(P_cur, min_score, max_per_layer), stamp_of(-1, L - 1, L))
    for t in range(n_tokens):
        prev = None
        for l in range(L):
            r = route(x_of(t, l), wg_of(l), K, renorm)
            rec["tie_boundary"] += int(r["tie_boundary"].sum())
            rec["tie_order"] += int(r["tie_order"].sum())
            cur = [sorted(int(v) for v in r["idx"][b]) for b in range(B)]
            psets = STPredictor.prefetch_sets(P_cur)
            rec["hits"][t, l] = sum(len(set(cur[b]) & set(psets[b])) for b in range(B))
            rec["npred"][t, l] = sum(len(p) for p in psets)
            rec["idx"].append(r["idx"])
            rec["w"].append(r["w"])
            pred.update(l, prev, cur, online=online)
            if l + 1 < L:
                P_next = pred.predict(l, cur, use_cct=use_cct, use_ht=use_ht)
            else:
                P_next = pred.predict(-1, None, use_cct=False, use_ht=use_ht)
            rec["scores"].append(P_next)
            if cache is not None:
                U = sorted(set(v for s in cur for v in s))
                cache.acquire(l, U, stamp_of(t, l, L))
            if ffn_of is not None and t < ffn_tokens:
                rec["y"][(t, l)] = ffn_of(l)(x_of(t, l), r["idx"], r["w"])
            if cache is not None and mode != MODE_ON_DEMAND:
                nl = (l + 1) % L
                cache.prefetch(nl, admitted(P_next, min_score, max_per_layer), stamp_of(t, l, L))
            prev, P_cur = cur, P_next
    rec["predictor"] = pred
    rec["cache"] = cache
    return rec
