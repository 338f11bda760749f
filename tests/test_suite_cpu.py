"""Host checks of the synthetic suite's case generator (no GPU): every case
is well formed, seeded draws are reproducible, and the value recipes hold
(constant values, zero upstream, shared key/value heads)."""
import numpy as np
import pytest

from synthetic import suite, bf16_bits_to_f32


def test_cases_are_well_formed():
    assert len(suite.CASES) >= 50
    for i, c in enumerate(suite.CASES):
        assert c.index == i
        assert c.Hq % c.Hkv == 0 and c.d in (64, 128)
        assert c.cu[0] == 0 and c.cu[-1] == c.total and np.all(np.diff(c.cu) >= 0)
        assert c.max_seqlen == max(c.lens) >= 1
        if not c.packed:
            assert len(set(c.lens)) == 1, "dense cases are B equal-length batches"
    cats = {c.category for c in suite.CASES}
    for need in ("packed", "unequal", "empty", "singleton", "tile boundary", "batch", "non-causal",
                 "key shift", "value shift", "constant values", "sharp", "zero upstream",
                 "tiny upstream", "long"):
        assert need in cats, need


@pytest.mark.parametrize("idx", [1, 14, 31, 38, 44])
def test_draws_reproducible_and_recipes_hold(idx):
    c = suite.CASES[idx]
    a, b = suite.make_case(c), suite.make_case(c)
    for n in ("q", "k", "v", "do"):
        assert np.array_equal(a[n], b[n])
    assert a["q"].shape == (c.Hq, c.total, c.d) and a["k"].shape == (c.Hkv, c.total, c.d)
    v = bf16_bits_to_f32(a["v"])
    if c.v_const:
        assert np.all(v == v[:, :1, :])
    if c.do_std == 0:
        assert np.all(bf16_bits_to_f32(a["do"]) == 0)
    other = suite.make_case(c, seed=7001)
    assert not np.array_equal(other["q"], a["q"])


def test_unequal_query_key_cases():
    cross = [c for c in suite.CASES if c.cross]
    assert len(cross) >= 8
    for c in cross:
        assert c.packed and len(c.lens_k) == len(c.lens)
        assert c.cu_k[0] == 0 and c.cu_k[-1] == c.total_k >= 1 and np.all(np.diff(c.cu_k) >= 0)
        assert c.max_seqlen_k == max(c.lens_k) >= 1
        x = suite.make_case(c)
        assert x["q"].shape == (c.Hq, c.total, c.d) and x["do"].shape == x["q"].shape
        assert x["k"].shape == (c.Hkv, c.total_k, c.d) and x["v"].shape == x["k"].shape
    # leading queries of a causal sequence with nq > nk see no key, and so
    # does every query of a sequence without keys
    more = next(c for c in cross if c.name == "more queries than keys")
    e = more.empty_rows()
    assert e.sum() == (100 - 40) + 0 + (130 - 2)
    assert e[:60].all() and not e[60:100].any() and e[170:298].all() and not e[298:].any()
    none = next(c for c in cross if c.name == "sequences without keys")
    assert none.empty_rows().sum() == 20 + 5
    nc = next(c for c in cross if c.name == "non-causal sequence without keys")
    assert nc.empty_rows().tolist() == [False] * 10 + [True] * 20
    nq0 = next(c for c in cross if c.name == "sequence without queries")
    assert nq0.unseen_keys().tolist() == [True] * 50 + [False] * 100
    assert not any(c.unseen_keys().any() for c in suite.CASES if c.name != nq0.name and c.cross)
    # square cases have no empty rows unless a sequence is empty
    assert not any(c.empty_rows().any() for c in suite.CASES if not c.cross)
