"""GPU tests of the best-kernel search module (apt_search_config): it picks a
config that runs, records it in the library's table, apt_select_config and
apt_gemm (cfg NULL) then use it, and results stay bit-exact; clearing the
table restores the model's choice."""
import numpy as np
import pytest

import paper_2508_19087_amd as apt
import synth
from gpu_util import assert_int32_equal, oracle_full, pack_problem, run

pytestmark = pytest.mark.gpu


@pytest.fixture
def clean_table():
    apt.apt_config_table_clear()
    yield
    apt.apt_config_table_clear()


def _same(c1, c2):
    return c1.as_dict() == c2.as_dict()


@pytest.mark.parametrize("M,N,K,p,q", [(1, 4096, 4096, 2, 2), (64, 300, 1000, 2, 4),
                                       (300, 513, 640, 3, 3), (129, 255, 1000, 8, 8)])
def test_search_records_and_is_used(clean_table, M, N, K, p, q):
    prob = synth.random_problem(synth.rng(4000, M, N, K, p, q), M, N, K, p, q)
    a, w = pack_problem(prob)
    model = apt.select_config(M, N, K, p, q)
    best, us = apt.search_config(a, w)
    assert us > 0
    assert apt.apt_config_table_size() == 1
    assert _same(apt.select_config(M, N, K, p, q), best)
    # a neighbouring problem is not in the table
    assert _same(apt.select_config(M + 1, N, K, p, q), apt.select_config(M + 1, N, K, p, q))
    want = oracle_full(prob)
    got, _ = run(prob, packed=(a, w))          # cfg NULL: the table's entry
    assert_int32_equal(got, want, "searched config")
    got, _ = run(prob, cfg=best, packed=(a, w))
    assert_int32_equal(got, want, "searched config, forced")
    apt.apt_config_table_clear()
    assert apt.apt_config_table_size() == 0
    assert _same(apt.select_config(M, N, K, p, q), model)


def test_search_prefill_shape(clean_table):
    """The W4A4 prefill shape: the searched config is at least as fast as the
    model's choice within timing noise, and exact on every output."""
    prob = synth.w4a4_prefill()
    a, w = pack_problem(prob)
    best, us = apt.search_config(a, w)
    assert best.route == apt.APT_ROUTE_INT8_MFMA
    got, _ = run(prob, packed=(a, w))
    assert_int32_equal(got, oracle_full(prob), "searched prefill")
