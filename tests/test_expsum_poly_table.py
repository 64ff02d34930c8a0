"""The fixed tables of the per-token polynomial of the quadrature's evaluation
(paper_2410_18234_amd/csrc/expsum_poly.h, written by gen_expsum_poly.py).

Checks that the committed header is what the generator writes, and that the
tables stand for what they claim, by evaluating them against the functions
directly: node term m, exp(-e^(m/2) x), within the recorded bound on
x in [1/4, e^(1/2)/4] (and the widened |t| <= 1.05); the expansion rows equal
(-e^(-1/2) x)^j; and a token's whole sum, nine node terms with coefficients
growing by up to e^(1/2) per node, within the stated relative bound.
"""
import importlib.util
import os
import re

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "..", "paper_2410_18234_amd", "csrc")


def _generator():
    spec = importlib.util.spec_from_file_location("gen_expsum_poly", os.path.join(CSRC, "gen_expsum_poly.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _table(text, name, rows, cols):
    body = text[text.index("__constant__ double " + name):]
    body = body[body.index("= {") + 3: body.index("};")]
    vals = [float(v) for v in re.findall(r"[-+]?[0-9][0-9.]*(?:e[-+]?[0-9]+)?", body)]
    assert len(vals) == rows * cols
    return np.array(vals).reshape(rows, cols)


def _header():
    with open(os.path.join(CSRC, "expsum_poly.h")) as f:
        return f.read()


def test_header_is_the_generator_output():
    text, _, _ = _generator().generate()
    assert _header() == text


def test_node_terms_and_expansion_rows():
    text = _header()
    g = _table(text, "kEsPolyG", 9, 11)
    h = _table(text, "kEsPolyH", 8, 11)
    xm = float(re.search(r"kEsPolyXm = ([0-9.eE+-]+);", text).group(1))
    dl = float(re.search(r"kEsPolyDelta = ([0-9.eE+-]+);", text).group(1))
    assert abs(xm - (0.25 + 0.25 * np.exp(0.5)) / 2) < 1e-15 and abs(dl - (0.25 * np.exp(0.5) - 0.25) / 2) < 1e-15
    t = np.random.default_rng(3).uniform(-1.05, 1.05, 50001)
    x = xm + dl * t
    for m in range(9):
        err = np.abs(np.polynomial.polynomial.polyval(t, g[m]) - np.exp(-np.exp(0.5 * m) * x)).max()
        assert err < 1e-10, (m, err)
    for j in range(8):
        assert np.allclose(np.polynomial.polynomial.polyval(t, h[j]), (-np.exp(-0.5) * x) ** j, rtol=1e-13, atol=1e-15)


def test_token_sum_relative_bound():
    # the bound the header states, for the largest growth c_(k+1) = e^(1/2) c_k and random decay
    text = _header()
    bound = float(re.search(r"below ([0-9.eE+-]+)\.", text).group(1))
    assert bound <= 5e-9
    g = _table(text, "kEsPolyG", 9, 11)
    xm = float(re.search(r"kEsPolyXm = ([0-9.eE+-]+);", text).group(1))
    dl = float(re.search(r"kEsPolyDelta = ([0-9.eE+-]+);", text).group(1))
    rng = np.random.default_rng(7)
    t = np.linspace(-1.0, 1.0, 4001)
    x = xm + dl * t
    e = np.exp(0.5 * np.arange(9))
    worst = 0.0
    for trial in range(200):
        decay = np.cumprod(np.concatenate([[1.0], rng.uniform(0.1, 1.0, 8)])) if trial else np.ones(9)
        c = e * decay
        exact = np.exp(-np.outer(x, e)) @ c
        approx = np.polynomial.polynomial.polyval(t, c @ g)
        worst = max(worst, np.abs(approx / exact - 1).max())
    assert worst <= bound, worst
