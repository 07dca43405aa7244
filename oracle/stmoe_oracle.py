"""Plain CPU oracle for the ST-MoE decode-step MoE layer.

TEST INFRASTRUCTURE.  Only the test suite, the package smoke check and the
benchmark's CPU-baseline leg may import or call this module.  The product path
never does, and this module imports nothing from the product package: it takes
the seeded input arrays as arguments and shares no code with the HIP path.

Arithmetic: float64 for every floating-point step, Python ints for the
prediction tables.  Each function names the passage of the paper it follows.

Parity status per function (see the pins under ``tests/``):
  router_logits / softmax_rows / topk_rows / route   pinned (invariants, brute force)
  swiglu_expert / moe_ffn                            pinned (explicit triple loop, special cases)
  STPredictor.profile / update / predict             pinned (hand-worked example, invariants,
                                                      closed form K^2/N, special cases)
  CacheSim                                           pinned (hand-worked trace, invariants,
                                                      exhaustive optimum lower bound)
  decode_reference (the per-layer loop)              pinned through its parts; its overall
                                                      hit rate on synthetic inputs has no
                                                      paper value: parity unpinned
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
    per-layer, per-batch-row History Table.

    cct_idx[i][e][s], cct_conf[i][e][s]: slot s of CCT entry e for the layer
    pair (i, i+1); ht[l][b]: the previous token's selection at layer l for
    batch row b, kept sorted ascending (it is a set).
    """

    def __init__(self, L: int, E: int, K: int, B: int = 1):
        self.L, self.E, self.K, self.B = L, E, K, B
        self.co = [[[0] * E for _ in range(E)] for _ in range(L - 1)]
        self.cct_idx = [[[0] * K for _ in range(E)] for _ in range(L - 1)]
        self.cct_conf = [[[0] * K for _ in range(E)] for _ in range(L - 1)]
        self.ht = [[[] for _ in range(B)] for _ in range(L)]

    # Algorithm 1 (and the HT initialisation of Section 4.1 / Fig. framework)
    def profile(self, sel) -> None:
        """sel[p][b][l][k]: the profiling tokens' selections.

        Co[i][e][f] counts, over all profiling tokens and batch rows, how often
        expert e at layer i and expert f at layer i+1 were selected together.
        CCT[i][e] keeps the K largest counts (ties and all-zero tails: lower
        index first) with confidence 2.  HT[l][b] is the last profiling token's
        selection.
        """
        sel = np.asarray(sel)
        P = sel.shape[0]
        for i in range(self.L - 1):
            co = self.co[i]
            for p in range(P):
                for b in range(self.B):
                    for e in sel[p, b, i]:
                        for f in sel[p, b, i + 1]:
                            co[int(e)][int(f)] += 1
            for e in range(self.E):
                order = sorted(range(self.E), key=lambda f: (-co[e][f], f))
                self.cct_idx[i][e] = order[:self.K]
                self.cct_conf[i][e] = [CONF_INIT] * self.K
        for l in range(self.L):
            for b in range(self.B):
                self.ht[l][b] = sorted(int(v) for v in sel[P - 1, b, l])

    # Algorithm 3 on one CCT entry
    def _update_entry(self, i: int, e: int, F) -> None:
        """Table update of one CCT entry e of pair i against the actual set F.

        Hit: confidence + 1, saturating at 3.  Miss: confidence - 1 while it is
        above 0; at 0 the slot is replaced by an expert of F that the entry did
        not hold before this update (candidates in ascending order, consumed one
        per replaced slot, slots visited in ascending order), with confidence 2.
        """
        row, conf = self.cct_idx[i][e], self.cct_conf[i][e]
        Fs = set(int(f) for f in F)
        fresh = sorted(Fs - set(row))
        nxt = 0
        for s in range(self.K):
            if row[s] in Fs:
                conf[s] = min(conf[s] + 1, CONF_MAX)
            elif conf[s] > 0:
                conf[s] -= 1
            else:
                row[s] = fresh[nxt]
                nxt += 1
                conf[s] = CONF_INIT

    def update(self, layer: int, prev_sets, cur_sets, online: bool = True) -> None:
        """Verify step at ``layer`` (Section 4.3.4): Algorithm 3 on CCT[layer-1]
        for every expert of the previous layer's selection, batch rows in order
        b = 0..B-1; then HT[layer][b] <- this token's selection."""
        if layer >= 1 and online:
            for b in range(self.B):
                for e in prev_sets[b]:
                    self._update_entry(layer - 1, int(e), cur_sets[b])
        for b in range(self.B):
            self.ht[layer][b] = sorted(int(v) for v in cur_sets[b])

    # Algorithm 2 + Eq. 1
    def predict(self, layer: int, cur_sets, use_cct: bool = True, use_ht: bool = True):
        """Scores for layer+1 from this token's selection at ``layer``.

        score_b[f] = sum over e in A_layer[b] of the confidence of f in CCT[layer][e]
                     + 2 if f is in HT[layer+1][b]                       (Eq. 1)
        layer == -1 predicts layer 0 from HT[0] alone (no earlier layer).
        Returns an int array [B][E].
        """
        tgt = layer + 1
        sc = np.zeros((self.B, self.E), dtype=np.int64)
        for b in range(self.B):
            if use_cct and layer >= 0:
                for e in cur_sets[b]:
                    for s in range(self.K):
                        sc[b, self.cct_idx[layer][int(e)][s]] += self.cct_conf[layer][int(e)][s]
            if use_ht:
                for f in self.ht[tgt][b]:
                    sc[b, f] += HT_SCORE
        return sc

    @staticmethod
    def prefetch_sets(scores):
        """Per-row PrefetchSet {f : score >= 2} (Algorithm 2)."""
        return [sorted(int(f) for f in np.nonzero(scores[b] >= THRESHOLD)[0])
                for b in range(scores.shape[0])]

    @staticmethod
    def ranked_union(scores):
        """Union of the rows' prefetch sets ranked by (max score desc, index asc)."""
        m = scores.max(axis=0)
        cand = [f for f in range(scores.shape[1]) if m[f] >= THRESHOLD]
        return sorted(cand, key=lambda f: (-int(m[f]), f))

    def tables(self):
        """(co [L-1][E][E], cct_idx [L-1][E][K], cct_conf [L-1][E][K], ht [L][B][K]) arrays."""
        return (np.array(self.co, np.int64).reshape(self.L - 1, self.E, self.E),
                np.array(self.cct_idx, np.int64).reshape(self.L - 1, self.E, self.K),
                np.array(self.cct_conf, np.int64).reshape(self.L - 1, self.E, self.K),
                np.array(self.ht, np.int64).reshape(self.L, self.B, self.K))


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
    """

    def __init__(self, L: int, E: int, C: int, warm=None):
        self.L, self.E, self.C = L, E, C
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
        return min(cands, key=lambda c: (self.last[l][c], c))

    def prefetch(self, l: int, ranked, stamp: int):
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
        for f in U:
            c = self._where(l, f)
            if c >= 0:
                self.n.hits += 1
                where[f] = c
                continue
            c = self._victim(l, keep)
            if c < 0:
                overflow.append(f)
                where[f] = -1
                continue
            self.slot[l][c] = f
            demand.append((f, c))
            where[f] = c
        for f, c in where.items():
            if c >= 0:
                self.last[l][c] = stamp
        self.n.demand += len(demand)
        self.n.overflow += len(overflow)
        self.n.useful += len(self.pending[l] & keep)
        self.n.wasted += len(self.pending[l] - keep)
        self.pending[l] = set()
        self.n.log.append(("A", l, stamp, tuple(demand), tuple(overflow)))
        return where, demand, overflow


# ----------------------------------------------------------------------------
# the per-layer decode loop (Section 4.3.4 workflow)
# ----------------------------------------------------------------------------

MODE_ON_DEMAND, MODE_STMOE, MODE_HT_ONLY, MODE_CCT_ONLY = 0, 1, 2, 3


def stamp_of(t: int, l: int, L: int) -> int:
    return t * L + l + 1


def decode_reference(L, E, K, B, x_of, wg_of, prof_sel, n_tokens, C=None, warm=None,
                     mode=MODE_STMOE, renorm=False, ffn_of=None, ffn_tokens=0, online=True):
    """Run the decode loop on the CPU.

    x_of(t, l) -> x [B][H] float64; wg_of(l) -> W_g [E][H] float64;
    ffn_of(l) -> callable(x, idx, w) -> y, used for the first ``ffn_tokens`` tokens.
    Per layer, in order: route; score this layer's prediction; Algorithm 3 on
    the previous layer pair and HT overwrite; predict the next layer (Eq. 1);
    demand-load the selection; FFN; prefetch the next layer's ranked set.
    online=False freezes the CCTs after profiling (Algorithm 3's confidence
    and replacement steps are skipped; HT is still overwritten).
    Returns a dict of per-(t, l) records and totals.
    """
    pred = STPredictor(L, E, K, B)
    pred.profile(prof_sel)
    use_cct = mode in (MODE_STMOE, MODE_CCT_ONLY)
    use_ht = mode in (MODE_STMOE, MODE_HT_ONLY)
    cache = CacheSim(L, E, C, warm) if C is not None else None
    # layer 0 of the first token is predicted from the profiled HT[0]
    P_cur = pred.predict(-1, None, use_cct=False, use_ht=use_ht)
    rec = dict(idx=[], w=[], scores=[], hits=np.zeros((n_tokens, L), np.int64),
               npred=np.zeros((n_tokens, L), np.int64), tie_boundary=0, tie_order=0, y={})
    if cache is not None and mode != MODE_ON_DEMAND:
        cache.prefetch(0, STPredictor.ranked_union(P_cur), stamp_of(-1, L - 1, L))
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
                cache.prefetch(nl, STPredictor.ranked_union(P_next), stamp_of(t, l, L))
            prev, P_cur = cur, P_next
    rec["predictor"] = pred
    rec["cache"] = cache
    return rec
