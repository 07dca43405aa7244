"""Pins of the oracle's decode loop (``decode_reference``): the order of the
per-layer steps of Section 4.3.4 (verify against this layer's prediction,
Algorithm 3 on the previous layer pair, HT overwrite, Eq. 1 for the next
layer with HT of that layer, missed loading, prefetch of the next layer) is
checked against hand-worked values, and planted slips in the oracle are shown
to fail those checks."""
import json
import os

import numpy as np
import pytest

import oracle.stmoe_oracle as O
from oracle.stmoe_oracle import (MODE_ON_DEMAND, MODE_STMOE, STPredictor, decode_reference,
                                 warm_from_profile)

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


G = _load("predictor_worked_example.json")
D = _load("decode_loop_worked_example.json")
E, K, L, B = G["E"], G["K"], G["L"], G["B"]
PROF = np.array([[[tok[0], tok[1]]] for tok in G["profiling"]])          # [P][B=1][L][K]
SEL = [(step["A0"], step["A1"]) for step in G["decode"]]


def _x_of(t, l):
    """One-hot hidden states: with the identity router the logits are 1 on
    the listed experts and 0 elsewhere, so top-K selects exactly that set."""
    x = np.zeros((B, E))
    x[0, SEL[t][l]] = 1.0
    return x


def _wg_of(l):
    return np.eye(E)


def _run(n_tokens, **kw):
    return decode_reference(L, E, K, B, _x_of, _wg_of, PROF, n_tokens, **kw)


def _pairs(pred):
    _, idx, conf, _ = pred.tables()
    return [[[int(idx[0, e, s]), int(conf[0, e, s])] for s in range(K)] for e in range(E)]


def _log(cache, full=False):
    out = []
    for ent in cache.n.log:
        if ent[0] == "P":
            out.append(["P", ent[1], ent[2], [list(c) for c in ent[3]]])
        else:
            out.append(["A", ent[1], ent[2], [list(c) for c in ent[3]], list(ent[4])] + (list(ent[5:]) if full else []))
    return out


def _counts(cache):
    n = cache.n
    return dict(hits=n.hits, demand=n.demand, overflow=n.overflow, prefetch=n.prefetch,
                useful=n.useful, wasted=n.wasted)


def mismatches_uncapped():
    """Every per-token value of the worked example that the loop reproduces
    differently (empty when the loop is right)."""
    bad = []
    T = len(G["decode"])
    rec = _run(T)
    for t, step in enumerate(G["decode"]):
        if rec["hits"][t, 0] != step["hits0"]:
            bad.append(("hits0", t))
        if rec["hits"][t, 1] != step["hits1"]:
            bad.append(("hits1", t))
        if rec["npred"][t, 0] != len(step["P0"]):
            bad.append(("npred0", t))
        if rec["npred"][t, 1] != len(step["P1"]):
            bad.append(("npred1", t))
        sc1 = rec["scores"][t * L + 0][0].tolist()
        if sc1 != step["scores1"]:
            bad.append(("scores1", t, sc1))
        # the prediction made at the last layer is next token's layer 0: HT[0] alone
        sc0 = rec["scores"][t * L + 1][0]
        if STPredictor.prefetch_sets(sc0[None])[0] != sorted(step["A0"]):
            bad.append(("next P0", t))
        # tables after this token (the loop is deterministic: a shorter run is a prefix)
        if _pairs(_run(t + 1)["predictor"]) != step["cct_after"]:
            bad.append(("cct_after", t))
    ht = rec["predictor"].tables()[3]
    if [ht[l][0].tolist() for l in range(L)] != G["final_ht"]:
        bad.append(("final_ht",))
    n = T * K
    if [int(rec["hits"][:, 0].sum()), n] != G["recall_l0"]:
        bad.append(("recall_l0",))
    if [int(rec["hits"][:, 1].sum()), n] != G["recall_l1"]:
        bad.append(("recall_l1",))
    if [int(rec["hits"][:, 1].sum()), int(rec["npred"][:, 1].sum())] != G["precision_l1"]:
        bad.append(("precision_l1",))
    return bad


def mismatches_capped(mode):
    cp = D["capped"]
    rec = _run(len(G["decode"]), C=cp["C"], warm=cp["warm"], mode=mode)
    key = "stmoe" if mode == MODE_STMOE else "on_demand"
    bad = []
    if _log(rec["cache"]) != cp[key + "_log"]:
        bad.append(("log", _log(rec["cache"])))
    if _counts(rec["cache"]) != cp[key + "_counts"]:
        bad.append(("counts", _counts(rec["cache"])))
    if mode == MODE_STMOE and rec["cache"].slot != cp["stmoe_final_slots"]:
        bad.append(("slots", rec["cache"].slot))
    return bad


def test_worked_example_through_the_loop():
    assert mismatches_uncapped() == []


def test_capped_loop_stmoe():
    assert mismatches_capped(MODE_STMOE) == []


def test_capped_loop_on_demand():
    assert mismatches_capped(MODE_ON_DEMAND) == []


def test_capped_loop_staged():
    """Staged prefetch inside the loop: the slots follow the on-demand trace
    exactly, the staged copies are the first non-resident ranked experts."""
    cp = D["capped"]
    rec = _run(len(G["decode"]), C=cp["C"], warm=cp["warm"], mode=MODE_STMOE, staged=2)
    assert _log(rec["cache"], full=True) == cp["staged2_log"]
    assert _counts(rec["cache"]) == cp["staged2_counts"]
    dem = _run(len(G["decode"]), C=cp["C"], warm=cp["warm"], mode=MODE_ON_DEMAND)
    assert rec["cache"].slot == dem["cache"].slot


def test_warm_start_policy():
    cp = D["capped"]
    assert warm_from_profile(PROF, L, E, cp["C"]).tolist() == cp["warm"]
    # more slots than experts: -1 padding
    assert warm_from_profile(PROF, L, E, 6)[0].tolist() == [0, 1, 2, 3, -1, -1]


def test_frozen_tables():
    """online=False: the CCT keeps its profiled contents, the HT still follows
    the selections, and the layer-1 predictions come from the frozen CCT."""
    fz = D["frozen"]
    T = len(G["decode"])
    rec = _run(T, online=False)
    assert _pairs(rec["predictor"]) == G["cct_after_profile"]
    ht = rec["predictor"].tables()[3]
    assert [ht[l][0].tolist() for l in range(L)] == fz["final_ht"]
    assert [rec["scores"][t * L][0].tolist() for t in range(T)] == fz["scores1"]
    assert rec["hits"][:, 1].tolist() == fz["hits1"]
    assert rec["npred"][:, 1].tolist() == fz["npred1"]
    # the layer-0 (temporal) part does not depend on the CCT
    assert rec["hits"][:, 0].tolist() == [s["hits0"] for s in G["decode"]]


def test_planted_tables_replace_profile():
    """tables=... replaces the profiled tables: zero confidences and an HT of
    experts never selected leave only score-0 predictions at token 0."""
    zero = np.zeros((L - 1, E, K), np.int64)
    idx = np.tile(np.arange(K), (L - 1, E, 1))
    ht = np.full((L, B, K), 0, np.int64)
    ht[:, :, :] = [2, 3]                   # token 0 selects {0,1} at layer 0: no overlap
    rec = _run(1, tables=(idx, zero, ht))
    assert rec["hits"][0, 0] == 0
    # layer 1 is scored from the zero-confidence CCT plus HT[1] = {2, 3}
    assert rec["scores"][0][0].tolist() == [0, 0, 2, 2]


# ---------------------------------------------------------------------------
# planted slips: each plausible mistake in the loop's order or indexing must
# fail one of the checks above.  The slips are planted in the oracle (on the
# CPU) with monkeypatch and undone after each test.
# ---------------------------------------------------------------------------

def _slip_predict_with_ht_of_this_layer(self, layer, cur_sets, use_cct=True, use_ht=True):
    sc = np.zeros((self.B, self.E), np.int64)
    for b in range(self.B):
        if use_cct and layer >= 0:
            for e in cur_sets[b]:
                for s in range(self.K):
                    sc[b, self.cct_idx[layer, int(e), s]] += self.cct_conf[layer, int(e), s]
        if use_ht:
            sc[b, self.ht[max(layer, 0), b]] += O.HT_SCORE
    return sc


def _slip_update_without_ht(orig):
    def f(self, layer, prev_sets, cur_sets, online=True):
        keep = self.ht[layer].copy()
        orig(self, layer, prev_sets, cur_sets, online)
        self.ht[layer] = keep
    return f


def _slip_update_wrong_pair(self, layer, prev_sets, cur_sets, online=True):
    # Algorithm 3 on the pair (layer, layer+1) instead of (layer-1, layer)
    if online and 1 <= layer and layer < self.L - 1:
        for b in range(self.B):
            for e in prev_sets[b]:
                self.update_entry(layer, int(e), cur_sets[b])
    for b in range(self.B):
        self.ht[layer, b] = sorted(int(v) for v in cur_sets[b])


def _slip_replacement_highest_first(self, i, e, F):
    row, conf = self.cct_idx[i, e], self.cct_conf[i, e]
    Fs = np.asarray(sorted(int(f) for f in F), np.int64)
    confirmed = np.isin(row, Fs)
    replaced = ~confirmed & (conf == 0)
    newcomers = np.setdiff1d(Fs, row)[::-1]
    conf[:] = np.where(confirmed, np.minimum(conf + 1, O.CONF_MAX), conf - 1)
    row[replaced] = newcomers[:int(replaced.sum())]
    conf[replaced] = O.CONF_INIT


def _slip_stamp(t, l, L_):
    return t * L_ + l


@pytest.mark.parametrize("slip", ["ht_of_this_layer", "no_ht_overwrite", "wrong_pair",
                                  "ht_score_1", "conf_cap_2"])
def test_planted_slip_fails_uncapped_pins(monkeypatch, slip):
    if slip == "ht_of_this_layer":
        monkeypatch.setattr(STPredictor, "predict", _slip_predict_with_ht_of_this_layer)
    elif slip == "no_ht_overwrite":
        monkeypatch.setattr(STPredictor, "update", _slip_update_without_ht(STPredictor.update))
    elif slip == "wrong_pair":
        monkeypatch.setattr(STPredictor, "update", _slip_update_wrong_pair)
    elif slip == "ht_score_1":
        monkeypatch.setattr(O, "HT_SCORE", 1)
    elif slip == "conf_cap_2":
        monkeypatch.setattr(O, "CONF_MAX", 2)
    assert mismatches_uncapped() != []


@pytest.mark.parametrize("slip", ["stamp", "prefetch_ht_of_this_layer", "threshold_3"])
def test_planted_slip_fails_capped_pins(monkeypatch, slip):
    if slip == "stamp":
        monkeypatch.setattr(O, "stamp_of", _slip_stamp)
    elif slip == "prefetch_ht_of_this_layer":
        monkeypatch.setattr(STPredictor, "predict", _slip_predict_with_ht_of_this_layer)
    elif slip == "threshold_3":
        monkeypatch.setattr(O, "THRESHOLD", 3)
    assert mismatches_capped(MODE_STMOE) != []


def test_planted_replacement_order_fails_double_replacement_pin(monkeypatch):
    """The worked example's only replacement has one candidate; the order in
    which several candidates fill replaced slots is pinned by the
    double-replacement example."""
    d = G["double_replacement"]

    def after():
        p = STPredictor(2, d["E"], d["K"], 1)
        p.cct_idx[0][0] = [s[0] for s in d["row"]]
        p.cct_conf[0][0] = [s[1] for s in d["row"]]
        p.update_entry(0, 0, d["F"])
        return [[int(p.cct_idx[0, 0, s]), int(p.cct_conf[0, 0, s])] for s in range(d["K"])]

    assert after() == d["after"]
    monkeypatch.setattr(STPredictor, "update_entry", _slip_replacement_highest_first)
    assert after() != d["after"]
