"""Host-side checks of the C-ABI library that need no GPU: it loads, exports
every entry point include/davet.h declares, rejects bad arguments before
enqueueing anything, and its host policy matches the oracle bit for bit."""

import math
import os
import re

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import paper_2608_01821_amd as dv
from oracle import policy as opol
from oracle import stats as ostats

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include",
                      "davet.h")


def test_exports_every_declared_symbol():
    text = open(HEADER).read()
    declared = set(re.findall(r"\b(davet_[a-z_0-9]+)\s*\(", text))
    assert declared, "no declarations found"
    lib = dv.raw()
    for name in sorted(declared):
        assert hasattr(lib, name), name
    assert declared <= set(dv.EXPORTED)
    assert "gfx950" in dv.davet_version()


def test_demand_prior_table(golden_dir):
    import json
    g = json.load(open(os.path.join(golden_dir, "table_a_demand_prior.json")))
    assert [dv.davet_demand_prior(i) for i in range(5)] == g["demand"]
    assert dv.davet_demand_prior(5) < 0 and dv.davet_demand_prior(-1) < 0


def _pol(B, rho, alpha, demand, early, K=3):
    return dv.Policy(B, rho, alpha, demand, 1 if early else 0, K)


@settings(max_examples=300, deadline=None)
@given(T=st.integers(1, 160), early=st.booleans(), B=st.floats(0.0, 1.2),
       rho=st.floats(0.0, 1.0), d=st.floats(0.0, 1.0),
       alpha=st.floats(0.0, 1.0), K=st.integers(1, 4), data=st.data())
def test_policy_bit_exact_vs_oracle(T, early, B, rho, d, alpha, K, data):
    pol = _pol(B, rho, alpha, d, early, K)
    lo, up = dv.davet_policy_envelope(pol, T)
    olo, oup = opol.envelope(T, early, B, rho, d)
    assert lo == olo and up == oup          # bitwise, element by element
    cb = data.draw(st.floats(0.0, 1.0))
    ch = data.draw(st.floats(0.0, 1.0))
    for t in range(1, T + 1):
        b, lv, r = dv.davet_policy_step(pol, t, T, lo, up, cb, ch)
        ob, olv, orr = opol.step(t, olo, oup, alpha, cb, ch, K)
        assert (b, lv, r) == (ob, olv, orr)


def test_policy_paper_defaults_closed_form():
    # Sec. 5.1 defaults; hand-derived levels (see the oracle's pins)
    pol = _pol(0.75, 0.20, 1.0, 1.0, True)
    lo, up = dv.davet_policy_envelope(pol, 16)
    assert up == [min(1.0, (33 - 2 * t) / 16) for t in range(1, 17)]
    lv = [dv.davet_policy_step(pol, t, 16, lo, up, 0.0, 0.0)[1]
          for t in range(1, 17)]
    assert "".join(map(str, lv)) == "2222222222211000"   # r = 1
    lv0 = [dv.davet_policy_step(pol, t, 16, lo, up, 1.0, 0.0)[1]
           for t in range(2, 17)]
    assert "".join(map(str, lv0)) == "222222111110000"    # r = 0 after t = 1


@settings(max_examples=200, deadline=None)
@given(data=st.data(), L=st.integers(0, 64), first=st.booleans())
def test_step_stats_bit_exact_vs_oracle(data, L, first):
    rng = np.random.default_rng(data.draw(st.integers(0, 2 ** 31)))
    conf = rng.random(L).astype(np.float32)
    am = rng.integers(0, 5, L).astype(np.int32)
    prev = rng.integers(0, 5, L).astype(np.int32)
    m = rng.integers(0, 2, L).astype(np.uint8)
    cb, ch = dv.davet_step_stats(conf, am, None if first else prev, m)
    assert cb == ostats.mean_conf(conf, m)
    assert ch == ostats.churn(am, prev, m, first)


@settings(max_examples=150, deadline=None)
@given(data=st.data(), L=st.integers(0, 1024), first=st.booleans(),
       power=st.sampled_from([1, 8, 24]))
def test_step_stats_bit_exact_vs_oracle_long(data, L, first, power):
    """Up to the library's largest response (1024 positions), with
    confidences spread over many binades (u^8, u^24) so that the float64
    sum's rounding depends on the order of its terms; exact zeros, ones and
    the smallest subnormal mixed in."""
    rng = np.random.default_rng(data.draw(st.integers(0, 2 ** 31)))
    conf = (rng.random(L) ** power).astype(np.float32)
    if L:
        special = np.array([0.0, 1.0, np.float32(1e-45), 0.5], np.float32)
        idx = rng.integers(0, L, min(L, 8))
        conf[idx] = special[rng.integers(0, 4, len(idx))]
    am = rng.integers(0, 126464, L).astype(np.int32)
    prev = np.where(rng.random(L) < 0.8, am,
                    rng.integers(0, 126464, L)).astype(np.int32)
    m = (rng.random(L) < data.draw(st.floats(0.0, 1.0))).astype(np.uint8)
    cb, ch = dv.davet_step_stats(conf, am, None if first else prev, m)
    assert cb == ostats.mean_conf(conf, m)
    assert ch == ostats.churn(am, prev, m, first)


def _expect(status, fn, *a, **k):
    with pytest.raises(dv.DavetError) as e:
        fn(*a, **k)
    assert e.value.status == status


def test_argument_validation_without_gpu():
    # every check below fails before any HIP call is made
    g = dv.ViewGeom(1, 12, 256, 3, dv.DAVET_F32)
    assert dv.davet_view_sizes(g) == [9, 36, 144]
    assert dv.davet_view_sizes(dv.ViewGeom(5, 27, 4096, 3, 1)) == \
        [245, 980, 3645]
    _expect(-2, dv.davet_view_sizes, dv.ViewGeom(1, 12, 256, 5, 0))
    _expect(-2, dv.davet_view_sizes, dv.ViewGeom(0, 12, 256, 3, 0))
    lib = dv.raw()
    import ctypes as C
    assert lib.davet_build_views(C.byref(g), None, None, None, None, None, 0,
                                 None) == -1
    bad = dv.ViewGeom(1, 12, 250, 3, dv.DAVET_F32)
    assert lib.davet_build_views(C.byref(bad), C.c_void_p(16), None, None,
                                 None, None, 0, None) == -2
    assert lib.davet_unmask(1, 32, 0, C.c_void_p(16), C.c_void_p(16),
                            C.c_void_p(16), C.c_void_p(16), None, None) == -1
    assert lib.davet_unmask(1, 2000, 2, C.c_void_p(16), C.c_void_p(16),
                            C.c_void_p(16), C.c_void_p(16), None, None) == -2
    cnt = C.c_int32(7)
    assert lib.davet_fp16_overflow_count(None, C.byref(cnt), None) == -1
    assert lib.davet_fp16_overflow_count(C.c_void_p(256), None, None) == -1
    assert lib.davet_fp16_overflow_count(C.c_void_p(16), C.byref(cnt),
                                         None) == -1
    assert cnt.value == 7
    assert lib.davet_set_attention_split(-1) == -1
    assert lib.davet_set_attention_split(9) == -1
    assert lib.davet_set_attention_split(0) == 0
    cfg = dv.ModelCfg(1, 4096, 32, 128, 12288, 126464, 126463, 1e-5, 1e4,
                      dv.DAVET_BF16)
    assert dv.davet_workspace_bytes(cfg, 1000, 1, 128) > 0
    badcfg = dv.ModelCfg(1, 4096, 32, 96, 12288, 126464, 126463, 1e-5, 1e4,
                         dv.DAVET_BF16)
    _expect(-2, dv.davet_workspace_bytes, badcfg, 1000, 1, 128)
    badcfg = dv.ModelCfg(1, 4096, 32, 128, 12288, 126464, 126464, 1e-5, 1e4,
                         dv.DAVET_BF16)
    _expect(-2, dv.davet_workspace_bytes, badcfg, 1000, 1, 128)
    badcfg = dv.ModelCfg(1, 4096, 32, 128, 12288, 126464, 5, 1e-5, 1e4, 7)
    _expect(-3, dv.davet_workspace_bytes, badcfg, 1000, 1, 128)
    _expect(-2, dv.davet_workspace_bytes, cfg, 1000, 65, 128)
    pol = _pol(0.75, 0.2, 1.0, 1.0, True)
    _expect(-1, dv.davet_policy_envelope, pol, 0)
    _expect(-1, dv.davet_policy_envelope, _pol(math.nan, 0.2, 1, 1, True), 4)
    lo, up = dv.davet_policy_envelope(pol, 4)
    _expect(-1, dv.davet_policy_step, pol, 5, 4, lo, up, 0.0, 0.0)
    _expect(-1, dv.davet_policy_step, _pol(0.75, 0.2, 1, 1, True, 9), 1, 4,
            lo, up, 0.0, 0.0)


def test_schedule_mailbox_and_wait_limit_checks():
    """Policy mode needs a caller-owned mailbox (the loop allocates nothing);
    the wait limit must be positive and finite.  No HIP call is made."""
    import ctypes as C
    lib = dv.raw()
    _expect(-1, dv.davet_set_wait_limit, 0.0)
    _expect(-1, dv.davet_set_wait_limit, -1.0)
    _expect(-1, dv.davet_set_wait_limit, math.inf)
    _expect(-1, dv.davet_set_wait_limit, math.nan)
    dv.davet_set_wait_limit(120.0)
    assert lib.davet_mailbox_create(None) == -1
    assert lib.davet_mailbox_destroy(None) == 0
    cfg = dv.ModelCfg(1, 256, 2, 128, 512, 1000, 999, 1e-5, 1e4,
                      dv.DAVET_F16)
    w = dv.WeightsT(16, 16, None, None, 0)
    g = (dv.ViewGeom * 1)(dv.ViewGeom(1, 7, 256, 3, dv.DAVET_F16))
    ptrs = (C.c_void_p * 2)(256, 256)
    cu = (C.c_int32 * 2)(0, 4)
    pol = (dv.Policy * 1)(_pol(0.75, 0.2, 1.0, 1.0, True))
    fixed = (C.c_int32 * 4)(0, 1, 2, 0)

    def call(pols, fixed_levels, T, mailbox):
        return lib.davet_run_schedule(
            C.byref(cfg), C.byref(w), 1, g, ptrs, ptrs, C.c_void_p(256), cu,
            8, T, 2, pols, fixed_levels, C.c_void_p(256), C.c_void_p(256),
            None, None, None, None, mailbox, C.c_void_p(256), 1 << 20, None)
    assert call(pol, None, 4, None) == -1
    assert "mailbox" in dv.raw().davet_last_error().decode()
    assert call(pol, fixed, 4, None) == -1      # both schedules given
    assert call(None, None, 4, None) == -1      # neither


def test_head_tiling_host_checks():
    """Tiled-head size formula and argument checks (no HIP call is made)."""
    import ctypes as C
    assert dv.davet_head_tiled_elems(126464, 4096) == 126464 * 4096
    assert dv.davet_head_tiled_elems(1000, 256) == 1024 * 256
    assert dv.davet_head_tiled_elems(1, 64) == 128 * 64
    assert dv.davet_head_tiled_elems(0, 64) == 0
    lib = dv.raw()
    a, b = C.c_void_p(1 << 20), C.c_void_p(1 << 30)
    assert lib.davet_pack_head(None, b, 1000, 256, dv.DAVET_F16, None) == -1
    assert lib.davet_pack_head(a, b, 1000, 256, dv.DAVET_F32, None) == -3
    assert lib.davet_pack_head(a, b, 1000, 100, dv.DAVET_F16, None) == -2
    assert lib.davet_pack_head(a, b, 0, 256, dv.DAVET_BF16, None) == -2
    # overlapping source and destination
    assert lib.davet_pack_head(a, C.c_void_p((1 << 20) + 4096), 1000, 256,
                               dv.DAVET_F16, None) == -1


def test_mixed_view_sizes_host():
    """Mixed-view token and member counts (Sec. 4.3 reading: coarse tokens
    plus the raw lattice o, o+S, ..., o = S/2), and geometry checks."""
    for C, G, S in [(1, 27, 2), (5, 27, 3), (2, 12, 4), (1, 1, 2), (3, 7, 5)]:
        lat = len(range(S // 2, G, S))
        g = dv.ViewGeom(C, G, 64, 3, dv.DAVET_BF16, S)
        n0 = -(-G // 4)
        n1 = -(-G // 2)
        assert dv.davet_view_sizes(g) == [C * n0 * n0, C * (n0 * n0 + lat * lat),
                                          C * G * G]
        assert dv.davet_view_map_sizes(g) == [C * G * G,
                                              C * (G * G + lat * lat), C * G * G]
        g0 = dv.ViewGeom(C, G, 64, 3, dv.DAVET_BF16)
        assert dv.davet_view_sizes(g0)[1] == C * n1 * n1
    for bad in (dv.ViewGeom(1, 27, 64, 4, 1, 2), dv.ViewGeom(1, 27, 64, 3, 1, 1),
                dv.ViewGeom(1, 27, 64, 3, 1, -2)):
        _expect(-2, dv.davet_view_sizes, bad)


def test_parse_operation_paper_examples(golden_dir):
    import json
    import os
    g = json.load(open(os.path.join(golden_dir,
                                    "table_operation_examples.json")))
    for q, cat in g["examples"]:
        assert dv.davet_parse_operation(q) == g["categories"][cat], q
    import ctypes as C
    assert dv.raw().davet_parse_operation(None, C.byref(C.c_int32())) == -1


_PARSER_WORDS = ["is", "are", "does", "can", "what", "which", "who", "where",
                 "how", "many", "much", "number", "of", "on", "the", "a",
                 "percentage", "%", "highest", "written", "text", "title",
                 "date", "when", "name", "country", "city", "company",
                 "shown", "image", "in", "this", "value", "<image>", "please",
                 "account", "counted", "more", "than", "say", "Question:",
                 "?", ",", "'s", "isn't", "answer", "with", "single",
                 "word", "or", "phrase", "IS", "Who", "HOW", "sum"]


@settings(max_examples=400, deadline=None)
@given(st.lists(st.sampled_from(_PARSER_WORDS), max_size=12),
       st.sampled_from([" ", "  ", "\n", "-", ""]))
def test_parse_operation_matches_oracle(words, sep):
    from oracle import parser
    q = sep.join(words)
    assert dv.davet_parse_operation(q) == parser.parse(q), q


def test_realizer_host_checks():
    # prune / merge keep the pooling counts; their map sizes and key counts
    # follow the documented formulas; every rejection happens before any HIP
    # call
    import ctypes as C
    lib = dv.raw()
    for rz in (dv.DAVET_REALIZER_PRUNE, dv.DAVET_REALIZER_MERGE):
        g = dv.ViewGeom(5, 27, 4096, 3, dv.DAVET_F16, 0, rz)
        assert dv.davet_view_sizes(g) == [245, 980, 3645]
        sizes = dv.davet_view_map_sizes(g)
        if rz == dv.DAVET_REALIZER_PRUNE:
            assert sizes == [245, 980, 3645]
            assert dv.davet_realizer_key_count(g) == 3645
        else:
            assert sizes == [3645, 3645, 3645]
            assert dv.davet_realizer_key_count(g) == 5 * 2 * 27 * 26
        assert dv.davet_views_scratch_bytes(g) > 8 * dv.davet_realizer_key_count(g)
        # grid above the limit, mixed view with another realizer
        _expect(-2, dv.davet_view_sizes, dv.ViewGeom(1, 65, 64, 3, 0, 0, rz))
        _expect(-2, dv.davet_view_sizes, dv.ViewGeom(1, 27, 64, 3, 0, 2, rz))
        # scratch missing or too small
        lv = (C.c_void_p * 2)(256, 256)
        assert lib.davet_build_views(C.byref(g), C.c_void_p(256), lv, None,
                                     None, None, 0, None) == -4
        assert lib.davet_build_views(C.byref(g), C.c_void_p(256), lv, None,
                                     None, C.c_void_p(256), 64, None) == -4
        # misaligned v
        assert lib.davet_build_views(C.byref(g), C.c_void_p(8), lv, None,
                                     None, None, 0, None) == -1
        assert lib.davet_realizer_keys(C.byref(g), C.c_void_p(8),
                                       C.c_void_p(256), None) == -1
    assert dv.davet_view_sizes(dv.ViewGeom(1, 64, 64, 3, 0, 0, 2)) == \
        [256, 1024, 4096]
    _expect(-1, dv.davet_view_sizes, dv.ViewGeom(1, 12, 64, 3, 0, 0, 3))
    pool = dv.ViewGeom(1, 12, 64, 3, 0)
    assert dv.davet_views_scratch_bytes(pool) == 0
    assert dv.davet_realizer_key_count(pool) == 0
    assert lib.davet_realizer_keys(C.byref(pool), C.c_void_p(256),
                                   C.c_void_p(256), None) == -1
    assert lib.davet_realizer_maps(C.byref(pool), C.c_void_p(256), None, None,
                                   None) == -1


def test_binding_refuses_strided_tensors():
    """The library reads every buffer as dense: the binding refuses a strided
    view instead of passing its storage address."""
    import torch
    from paper_2608_01821_amd import _lib
    x = torch.zeros(4, 6)
    assert _lib._ptr(x).value == x.data_ptr()
    assert _lib._ptr(None) is None
    with pytest.raises(ValueError):
        _lib._ptr(x.t())
    with pytest.raises(ValueError):
        _lib._ptr_array([x, x[:, 1]])
    lw = dict(wqkv=x, wo=x, wg=x, wu=x, wd=x.t())
    with pytest.raises(ValueError):
        dv.Weights(x, x, [lw])
