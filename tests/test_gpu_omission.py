"""The differential omission test (section 5.4, Eq. 4) on the GPU, through the C ABI: the collision
matrix must equal the oracle's on a small ragged case, and at the benchmark's size it must show
the closed-form pattern (withheld dimension: every block coincides; bound: none), with sampled
per-request hit lengths equal to the oracle's coinciding-block counts."""

import numpy as np
import pytest

from oracle.omission import equal_blocks, omission_matrix, project, vary
from tests.gpu_util import announce, gpu_available
from workloads import make_omission, make_omission_tiny

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X GPU")]


@pytest.fixture(scope="module")
def pkv():
    import paper_2609_38706_amd as m
    m.lib()
    return m


def test_omission_matrix_matches_oracle(pkv):
    from paper_2609_38706_amd.omission import omission_check
    announce("omission-tiny: GPU vs oracle")
    case = make_omission_tiny()
    want = omission_matrix(case, threads=4)
    got = omission_check(case)
    assert got["blocks"] == want["blocks"]
    assert (got["collisions"] == want["collisions"]).all()
    assert (got["omission"] == want["omission"]).all()


def test_declared_change_gates_the_report_on_gpu(pkv):
    from paper_2609_38706_amd.omission import omission_check
    case = make_omission_tiny()
    case.changes = {d: d != b"salt" for d in case.dims}
    got = omission_check(case)
    j = case.dims.index(b"salt")
    assert not got["omission"][:, j].any()
    assert (got["omission"] == omission_matrix(case)["omission"]).all()


def test_omission_pattern_at_benchmark_size(pkv):
    from paper_2609_38706_amd.omission import OmissionRun
    announce("omission: 512 x 1024 tokens, 20 dimensions, 22 bindings")
    case = make_omission()
    run = OmissionRun(case)
    run.run()
    res = run.result()
    blocks = res["blocks"]
    assert blocks == case.batch.n_req * 1024 // 16
    for i, (label, names) in enumerate(case.bindings):
        for j, d in enumerate(case.dims):
            bound = names is None or d in names
            assert res["collisions"][i, j] == (0 if bound else blocks), (label, d)
    # sampled: per-request hit lengths of a few groups against the oracle on the first 8 requests
    b = case.batch
    sub = slice(0, 8)
    toks = b.tokens[: int(b.tok_off[8])]
    off = b.tok_off[:9]
    base = b.request_descs()[sub]
    for i, j in [(0, 0), (1, 0), (5, 4), (len(case.bindings) - 1, 19)]:
        names = case.bindings[i][1]
        dim = case.dims[j]
        want = equal_blocks(toks, off, b.block, [project(d, names) for d in base],
                            [project(vary(d, dim, case.variants[dim]), names) for d in base], threads=4)
        assert (run.variant_hits(i, j)[:8] == want).all(), (i, j)
