"""Pins of the oracle's bfloat16 rounding points.

In bf16 mode the oracle rounds to bfloat16 (round-to-nearest-even):
  * the input rows X (batch gradient, SGD steps, prediction);
  * the weights, each time they serve as a GEMM operand: the forward product
    and the backward product G_l W_l^T;
  * each hidden activation after ReLU;
  * each gradient G_l before it serves as an operand (of dW_l and G_{l-1}).
A hidden layer's bias gradient is the column sum of that rounded G_l, the
output layer's the column sum of the unrounded one.

Each check below runs a hand-built net in which exactly one of these values
is not representable in bfloat16 while every other operand is, so no other
rounding fires.  The expected loss or gradient follows from the definition
(softmax cross-entropy, dW = A^T G, G_{l-1} = G_l W_l^T) with that one value
rounded.  The rounding in the expectations is torch's float32 -> bfloat16
conversion, not the oracle's.  ``test_each_rounding_point_is_pinned`` builds
the oracle once per rounding point with that point removed and checks that
some check here fails: a dropped rounding cannot pass unnoticed.
"""
import json
import math
import os
import re
import subprocess
import sys
import tempfile

import numpy as np
import pytest
import torch

import oracle

E10, E11, E9 = 2.0 ** -10, 2.0 ** -11, 2.0 ** -9


def bf(x: float) -> float:
    """float32 -> bfloat16 (round-to-nearest-even) -> float, via torch."""
    return float(torch.tensor([x], dtype=torch.float32).to(torch.bfloat16).float().item())


def f32(x: float) -> float:
    return float(np.float32(x))


def sigmoid(z: float) -> float:
    return 1.0 / (1.0 + math.exp(-z))


def assert_off_tie(x: float):
    """x is well away from a bfloat16 rounding boundary (so binary32 noise in
    the oracle's value cannot change its rounding)."""
    m, e = math.frexp(abs(x))                      # x = m 2^e, m in [0.5, 1)
    frac = (m * 256.0) % 1.0                       # position between bf16 neighbours
    assert 0.05 < abs(frac - 0.5) < 0.45, x


def close(a, b, rel=1e-6):
    return abs(a - b) <= rel * max(abs(b), 1e-30)


# net 1 -> 2 with W = [w0, w1], b = 0: logits (x w0, x w1)
def _p12(w0, w1):
    return np.array([w0, w1, 0.0, 0.0])


# net 1 -> 1 -> 2: W1 = [w1], b1 = [b1], W2 = [u0, u1], b2 = 0
def _p112(w1, b1, u0, u1):
    return np.array([w1, b1, u0, u1, 0.0, 0.0])


CE_ONE_ZERO = math.log(1.0 + math.e)               # CE of logits (1, 0), label 1
X1 = np.array([[1.0]], np.float32)
Y1 = np.array([1], np.int32)


def check_x_batch_grad():
    """X = 1 + 2^-10 rounds to 1: logits (1, 0), CE = log(1 + e)."""
    x = np.array([[1.0 + E10]], np.float32)
    assert bf(float(x[0, 0])) == 1.0
    ce, _, _, _ = oracle.batch_grad("bf16", [1, 2], _p12(1.0, 0.0), x, Y1)
    assert close(ce, CE_ONE_ZERO), (ce, CE_ONE_ZERO)


def check_x_train_steps():
    """The loss of an SGD step (taken before the update) sees bf16(X)."""
    x = np.array([[1.0 + E10]], np.float32)
    params = _p12(1.0, 0.0).copy()
    ce, _ = oracle.train_steps("bf16", [1, 2], params, np.ones(2, np.uint8), 0.0, x, Y1,
                               np.zeros(1, np.uint32), 1, 0, 1)
    assert close(ce, CE_ONE_ZERO), (ce, CE_ONE_ZERO)


def check_x_predict():
    x = np.array([[1.0 + E10]], np.float32)
    ce, corr = oracle.predict("bf16", [1, 2], _p12(1.0, 0.0), x, Y1)
    assert close(ce, CE_ONE_ZERO), (ce, CE_ONE_ZERO)
    assert corr == 0                               # argmax is class 0


def check_w_forward():
    """W = (1 + 2^-10, 0) rounds to (1, 0) in the forward product."""
    ce, _, _, _ = oracle.batch_grad("bf16", [1, 2], _p12(1.0 + E10, 0.0), X1, Y1)
    assert close(ce, CE_ONE_ZERO), (ce, CE_ONE_ZERO)


def check_relu_activation():
    """Z1 = 1 + 2^-10 (the bias is not an operand): A1 = bf16(Z1) = 1."""
    ce, _, _, _ = oracle.batch_grad("bf16", [1, 1, 2], _p112(1.0, E10, 1.0, 0.0), X1, Y1)
    assert close(ce, CE_ONE_ZERO), (ce, CE_ONE_ZERO)


def check_output_gradient_operand():
    """Logits (1, 0), label 1, b = 1: G = (p0, p1 - 1) = (s, -s) with
    s = sigmoid(1).  dW = x^T bf16(G); the output bias gradient is the
    unrounded column sum."""
    s = sigmoid(1.0)
    g = f32(s)
    assert_off_tie(g)
    _, grads, _, _ = oracle.batch_grad("bf16", [1, 2], _p12(1.0, 0.0), X1, Y1)
    dW, db = grads[:2], grads[2:]
    assert dW[0] == bf(g) and dW[1] == -bf(g), (dW, bf(g))
    assert close(db[0], s) and close(db[1], -s), (db, s)


def check_w_backward():
    """W2 = (1 + 2^-10, 1 + 2^-11): both round to 1, the logits tie, G2 =
    (1/2, -1/2) exactly, and G1 = G2 bf16(W2)^T = 0 (unrounded it would be
    2^-12)."""
    _, grads, _, _ = oracle.batch_grad("bf16", [1, 1, 2], _p112(1.0, 0.0, 1.0 + E10, 1.0 + E11), X1, Y1)
    dW1, db1, dW2, db2 = grads[0], grads[1], grads[2:4], grads[4:6]
    assert dW1 == 0.0 and db1 == 0.0, (dW1, db1)
    assert list(dW2) == [0.5, -0.5] and list(db2) == [0.5, -0.5], (dW2, db2)


def check_hidden_gradient_and_bias():
    """W2 = (1, 2^-9): G2 = (s, -s) with s = sigmoid(1 - 2^-9);
    G1 = bf16(s) (1 - 2^-9), not bf16-representable.  The hidden layer's dW1
    and db1 both take bf16(G1); the output layer's db2 takes the unrounded G2."""
    s = sigmoid(1.0 - E9)
    g2 = bf(f32(s))
    assert_off_tie(f32(s))
    g1 = f32(g2 * (1.0 - E9))
    assert_off_tie(g1)
    want = bf(g1)
    assert want != g1
    _, grads, _, _ = oracle.batch_grad("bf16", [1, 1, 2], _p112(1.0, 0.0, 1.0, E9), X1, Y1)
    dW1, db1, dW2, db2 = grads[0], grads[1], grads[2:4], grads[4:6]
    assert dW1 == want and db1 == want, (dW1, db1, want, g1)
    assert dW2[0] == g2 and dW2[1] == -g2, (dW2, g2)
    assert close(db2[0], s) and close(db2[1], -s), (db2, s)


CHECKS = [check_x_batch_grad, check_x_train_steps, check_x_predict, check_w_forward, check_relu_activation,
          check_output_gradient_operand, check_w_backward, check_hidden_gradient_and_bias]


@pytest.mark.parametrize("check", CHECKS, ids=[c.__name__ for c in CHECKS])
def test_rounding_point(check):
    check()


def test_f32_mode_rounds_none_of_them():
    """Sanity of the constructions: in f32 mode the same nets see the
    unrounded values, so every one of the checks above would fail there."""
    x = np.array([[1.0 + E10]], np.float32)
    ce, _, _, _ = oracle.batch_grad("f32", [1, 2], _p12(1.0, 0.0), x, Y1)
    want = math.log(1.0 + math.exp(1.0 + E10))
    assert close(ce, want) and not close(ce, CE_ONE_ZERO)
    _, grads, _, _ = oracle.batch_grad("f32", [1, 1, 2], _p112(1.0, 0.0, 1.0 + E10, 1.0 + E11), X1, Y1)
    assert grads[0] != 0.0


def run_checks():
    """Names of the checks that fail (used by the mutation test below)."""
    failed = []
    for c in CHECKS:
        try:
            c()
        except AssertionError:
            failed.append(c.__name__)
    return failed


# ----------------------------------------------------------- mutation check
def _rop_sites(src: str):
    """(start, end, inner) of every ``rop(mode, EXPR)`` call in the source."""
    out = []
    for m in re.finditer(r"\brop\(mode, ", src):
        depth, i = 1, m.end()
        while depth:
            depth += {"(": 1, ")": -1}.get(src[i], 0)
            i += 1
        out.append((m.start(), i, src[m.end():i - 1]))
    return out


def _mutants(src: str):
    muts = []
    for k, (a, b, inner) in enumerate(_rop_sites(src)):
        line = src.count("\n", 0, a) + 1
        muts.append((f"rop at line {line}", src[:a] + "(" + inner + ")" + src[b:]))
    db = "(l == L ? G : Gop)"
    assert src.count(db) == 1
    muts.append(("hidden db from the unrounded G", src.replace(db, "G")))
    muts.append(("output db from the rounded G", src.replace(db, "Gop")))
    return muts


def test_each_rounding_point_is_pinned():
    src_path = os.path.join(os.path.dirname(oracle.__file__), "gevo_oracle.c")
    with open(src_path) as f:
        src = f.read()
    muts = _mutants(src)
    assert len(muts) == 9                          # seven rop() sites plus the two bias-gradient readings
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    survivors = []
    with tempfile.TemporaryDirectory() as d:
        for k, (name, msrc) in enumerate(muts):
            c = os.path.join(d, f"m{k}.c")
            so = os.path.join(d, f"m{k}.so")
            with open(c, "w") as f:
                f.write(msrc)
            subprocess.run(["gcc", "-O1", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
                            "-o", so, c, "-lm"], check=True)
            code = ("import sys, json; sys.path.insert(0, sys.argv[1]); import oracle; oracle._LIB_PATH = sys.argv[2];"
                    "from tests import test_oracle_bf16_points as t; print(json.dumps(t.run_checks()))")
            res = subprocess.run([sys.executable, "-c", code, root, so], capture_output=True, text=True, timeout=300)
            assert res.returncode == 0, res.stderr[-2000:]
            failed = json.loads(res.stdout.strip().splitlines()[-1])
            if not failed:
                survivors.append(name)
    assert not survivors, f"rounding points no check detects: {survivors}"
