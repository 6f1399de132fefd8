"""Oracle on the tiny synthetic decode workload, plus its independence.

Method quality (needle recall, agreement with full attention) is a property
of BinaryPC on these synthetic keys, not something the paper pins on them:
it is reported here, and only the default-needle recall (which the oracle
reaches exactly) is asserted.
"""

import ast
import os

import numpy as np
import pytest

import oracle as o
from _helpers import bits_of
from workloads import CONFIGS, make_layer

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(mode):
    cfg = CONFIGS[0]
    d = make_layer(cfg, device="cpu", needle_mode=mode)
    K, V, q = bits_of(d["K"]), bits_of(d["V"]), bits_of(d["q"])
    G = d["G"].numpy()
    pos = d["needle_pos"].numpy()
    sm = 1.0 / np.sqrt(cfg.D)
    rec, rec_exact, cos = [], [], []
    for h in range(cfg.Hkv):
        P, codes, err, fr = o.build_binary_pcs(K[0, h], G)
        qg = q[0, h * cfg.G:(h + 1) * cfg.G]
        r = o.decode_head(qg, K[0, h], V[0, h], codes, P, cfg.k, sm)
        assert r["idx"].shape == (cfg.k,) and np.all(np.diff(r["idx"]) > 0)
        full = o.full_attention(qg, K[0, h], V[0, h], sm)
        rec.append(np.isin(pos[0, h], r["idx"]).mean())
        rec_exact.append(np.isin(pos[0, h], o.exact_topk(qg, K[0, h], cfg.k)).mean())
        num = (r["out"] * full).sum(axis=1)
        cos.append(float(np.mean(num / np.linalg.norm(r["out"], axis=1) / np.linalg.norm(full, axis=1))))
    return float(np.mean(rec)), float(np.mean(rec_exact)), float(np.mean(cos))


def test_needle_recall_default():
    rec, rec_exact, cos = _run("rho")
    print(f"needles 3*rho*q/|q|: hash recall {rec:.3f}, exact-top-k recall {rec_exact:.3f}, cos {cos:.5f}")
    assert rec_exact == 1.0 and rec == 1.0


@pytest.mark.slow
@pytest.mark.parametrize("mode", ["literal", "q3"])
def test_needle_variants_reported(mode):
    rec, rec_exact, cos = _run(mode)
    print(f"needles {mode}: hash recall {rec:.3f}, exact-top-k recall {rec_exact:.3f}, cos {cos:.5f}")


def test_oracle_imports_nothing_of_the_product():
    allowed = {"numpy", "__future__"}
    for fn in os.listdir(os.path.join(ROOT, "oracle")):
        if not fn.endswith(".py"):
            continue
        tree = ast.parse(open(os.path.join(ROOT, "oracle", fn)).read())
        for node in ast.walk(tree):
            if isinstance(node, ast.Import):
                names = [a.name.split(".")[0] for a in node.names]
            elif isinstance(node, ast.ImportFrom):
                if node.level:  # relative import inside the oracle package
                    continue
                names = [node.module.split(".")[0]]
            else:
                continue
            assert set(names) <= allowed, (fn, names)


def test_generator_imports_neither_side():
    # the shared input module may import neither the oracle nor the HIP package
    for fn in os.listdir(os.path.join(ROOT, "workloads")):
        if not fn.endswith(".py"):
            continue
        tree = ast.parse(open(os.path.join(ROOT, "workloads", fn)).read())
        for node in ast.walk(tree):
            if isinstance(node, ast.Import):
                names = [a.name.split(".")[0] for a in node.names]
            elif isinstance(node, ast.ImportFrom) and not node.level:
                names = [node.module.split(".")[0]]
            else:
                continue
            assert not set(names) & {"oracle", "paper_2608_04405_amd"}, (fn, names)
