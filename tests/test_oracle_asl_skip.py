"""Pins of the ASL-Skip oracle (Sec. 4.2-4.3, Alg. 1, Eq. 4-6, Table 10)."""
import json
import os

import numpy as np
import pytest

from oracle import asl_skip as ak
from synth.skip_inputs import REPLACED_LAYERS, slc_tables, policy_lists

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_table10_lists_partition_layers_and_match_text_claims():
    claims = json.load(open(os.path.join(GOLDEN, "replaced_layers_claims.json")))
    for name, lists in REPLACED_LAYERS.items():
        c = claims[name]
        allv = list(lists["attn"]) + list(lists["ffn"])
        assert sorted(allv) == list(range(c["L"]))
        assert len(lists["ffn"]) == c["n_ffn"]
        assert lists["attn"][0] == c["first_attn"] and lists["ffn"][0] == c["first_ffn"]


@pytest.mark.parametrize("name", ["llava15_7b", "llava_next_7b", "synthetic_40"])
def test_eq5_and_argmax_reproduce_lists(name):
    L = 40 if name == "synthetic_40" else 32
    lists = policy_lists(name, L)
    sa, sf = slc_tables(lists, L)
    na, nf = ak.slc_normalize(sa, sf)
    m, sel = ak.skip_targets(na, nf)
    assert [l for l in range(L) if m[l] == ak.ATTN] == sorted(lists["attn"])
    assert [l for l in range(L) if m[l] == ak.FFN] == sorted(lists["ffn"])
    # each list is in order of decreasing normalised score of the designated module
    for key, fam in (("attn", na), ("ffn", nf)):
        vals = [fam[l] for l in lists[key]]
        assert all(vals[i] > vals[i + 1] for i in range(len(vals) - 1))


def test_eq5_extremes():
    na, nf = ak.slc_normalize([0.5, 0.2, 0.9], [3.0, 3.0, 1.0])
    assert na[1] == pytest.approx(1.0) and na[2] == pytest.approx(0.0, abs=1e-7)
    assert na[0] == pytest.approx(1 - 0.3 / 0.7, abs=1e-7)
    assert nf[2] == pytest.approx(1.0) and nf[0] == pytest.approx(0.0, abs=1e-7)


def test_target_tie_goes_to_attention():
    m, sel = ak.skip_targets([0.5, 0.7, 0.2], [0.5, 0.1, 0.9])
    assert list(m) == [ak.ATTN, ak.ATTN, ak.FFN]
    assert list(sel) == [0.5, 0.7, 0.9]


def test_eq4_skippability():
    assert ak.skippability(0.2, 0.3) == pytest.approx(0.5)
    assert ak.skippability(0.7, 0.6) == 0.0
    assert ak.skippability(0.0, 0.0) == 1.0


def test_entropy_normalisation_extremes():
    W = np.eye(8) * 200.0
    assert ak.entropy_norm(np.zeros((1, 8)), W)[0] == pytest.approx(1.0)
    assert ak.entropy_norm(np.eye(8)[:1], W)[0] == pytest.approx(0.0, abs=1e-6)
    # two equally likely words out of V=4: ln 2 / ln 4 = 1/2
    W2 = np.array([[1.0, 0], [1.0, 0], [0, 0], [0, 0]]) * 100.0
    assert ak.entropy_norm(np.array([[1.0, 0.0]]), W2)[0] == pytest.approx(0.5, abs=1e-6)


def test_itc_extremes():
    t = np.array([[1.0, 0.0], [3.0, 0.0]])
    hv = np.array([[2.0, 0.0], [-1.0, 0.0], [0.0, 5.0], [0.0, 0.0]])
    assert list(ak.itc(hv, t)) == pytest.approx([1.0, 0.0, 0.5, 0.5])


def test_plan_hand_table():
    # window = L//2 = 2 layers; w1 = w2 = 1, T_skip = 1.5
    S_sa = np.array([[1.0, 0.2, 0.0],
                     [0.0, 0.9, 0.3]], np.float32)
    slc_sel = [0.5, 0.5, 1.0, 1.0]
    m = [ak.ATTN, ak.FFN, ak.ATTN, ak.ATTN]
    codes, admit, target = ak.plan(S_sa, slc_sel, m, 1.0, 1.0, 1.5, 4)
    # token 0 reaches exactly 1.5 at layer 0 (">=" admits) -> attention from layer 0
    # token 1: 0.7, then 2.1 at layer 1 -> target frozen to m(1) = FFN from layer 1
    # token 2: 0.5, then 1.3; the window closes before layer 2
    assert list(admit) == [0, 1, -1]
    assert list(target) == [ak.ATTN, ak.FFN, -1]
    assert codes.tolist() == [[1, 0, 0], [1, 2, 0], [1, 2, 0], [1, 2, 0]]


def test_plan_target_frozen_and_accumulation_stops():
    L = 8
    S_sa = np.ones((4, 1), np.float32)
    m = [ak.FFN, ak.ATTN, ak.ATTN, ak.ATTN, ak.FFN, ak.FFN, ak.FFN, ak.FFN]
    codes, admit, target = ak.plan(S_sa, [1.0] * L, m, 1.0, 1.0, 2.0, L)
    assert admit[0] == 0 and target[0] == ak.FFN
    assert codes[:, 0].tolist() == [2] * L
    # a threshold reachable only after the window never admits
    codes, admit, _ = ak.plan(S_sa, [1.0] * L, m, 1.0, 1.0, 8.5, L)
    assert admit[0] == -1 and codes.sum() == 0


def test_plan_weights():
    # w1 = 3, w2 = 1: 3*0.5 + 1*0.5 = 2 per layer -> reaches 4 at layer 1
    codes, admit, _ = ak.plan(np.full((5, 1), 0.5, np.float32), [0.5] * 10, [0] * 10,
                              3.0, 1.0, 4.0, 10)
    assert admit[0] == 1


def test_pack_codes_text_rows_zero():
    c = [np.full((2, 5), 3, np.uint8), np.full((2, 5), 1, np.uint8)]
    p = ak.pack_codes(c, [3, 2], 2, 2)
    assert p.shape == (2, 3 + 2 + 2 + 2)
    assert p[0].tolist() == [3, 3, 3, 0, 0, 1, 1, 0, 0]
