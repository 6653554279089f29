"""The seeded generator: determinism, head-subset independence, bf16 exactness, plants."""
import numpy as np

from synth import gen as G


def test_deterministic_and_subset_independent():
    a = G.make_layer(2, n=512)
    b = G.make_layer(2, n=512, q_heads=[5], kv_heads=[1])
    assert np.array_equal(a["q"][5], b["q"][5]) and np.array_equal(a["k"][1], b["k"][1])
    assert np.array_equal(a["v"][1], b["v"][1])
    assert not b["q"][4].any()


def test_bf16_exact_and_rounding():
    a = G.make_layer(2, n=256)
    for x in (a["q"], a["k"], a["v"]):
        assert np.array_equal(G.bf16_round(x), x)
    x = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5], dtype=np.float32)
    assert G.bf16_round(x).tolist() == [1.0, 1.0 + 2 ** -6, -2.5]   # ties to even


def test_planted_sink_dominates_logits():
    a = G.make_layer(1)
    q, k = a["q"][0].astype(np.float64), a["k"][0].astype(np.float64)
    lg = q[-64:] @ k.T / np.sqrt(64)
    spec = a["spec"]
    cols = spec.groups[0].vert_cols
    other = np.setdiff1d(np.arange(4, 2048), cols)
    assert lg[:, :4].mean() > lg[:, other].mean() + 3.0
    assert lg[:, cols].mean() > lg[:, other].mean() + 2.0


def test_evidence_spans_and_regimes():
    s = G.layer_spec(4)
    assert s.span_starts.size == 8
    assert np.all(s.span_starts[1:] > s.span_starts[:-1])
    ok = s.chunk_span >= 0
    assert np.all(s.span_starts[s.chunk_span[ok]] < np.nonzero(ok)[0] * 1024)
    regs = [G.layer_spec(5, l).groups[0].regime for l in range(32)]
    assert set(regs) <= set(G.REGIMES) and len(set(regs)) >= 3
