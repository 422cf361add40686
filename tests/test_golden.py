"""The oracle still reproduces its frozen output on the tiny workload
(tests/golden/tiny_oracle.txt, written by tests/golden/make_golden.py)."""
import os

import numpy as np

import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tiny_oracle.txt")


def _parse():
    heads = []
    for line in open(GOLDEN):
        if line.startswith("#"):
            continue
        tok = line.split()
        if tok[0] == "head":
            heads.append({"kv_len": int(tok[3]), "rows": {}})
        elif tok[0] == "kept":
            heads[-1]["kept"] = [int(v) for v in tok[1:]]
        elif tok[0] == "scores_hex":
            heads[-1]["scores"] = np.array([int(v, 16) for v in tok[1:]], np.uint32)
        elif tok[0] == "row":
            heads[-1]["rows"][int(tok[1])] = (float(tok[3]), np.array([float(v) for v in tok[5:]]))
    return heads


def test_oracle_matches_golden(oracle_lib):
    gold = _parse()
    cfg = W.tiny_config()
    x = W.make_layer_inputs(cfg, seed=0)
    rows = sorted(gold[0]["rows"])
    r = oracle.run_layer(cfg, x, rows=np.array(rows, np.int32))
    for h, g in enumerate(gold):
        assert int(r.kv_len[h]) == g["kv_len"]
        assert r.kept_seg[h].tolist() == g["kept"]
        np.testing.assert_array_equal(r.scores[h].view(np.uint32), g["scores"])
        for i, row in enumerate(rows):
            lse, o = g["rows"][row]
            np.testing.assert_allclose(r.lse[h, i], lse, rtol=0, atol=1e-13)
            np.testing.assert_allclose(r.O[h, i], o, rtol=0, atol=1e-13)
