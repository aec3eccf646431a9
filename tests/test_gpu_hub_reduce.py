"""The hub-row reduction on both of its kernels.

Rows of degree above deg_bound are cut into chunks of H nonzeros, each chunk
writes a partial row, and one more kernel adds a row's partials (Sec. III-C,
the hub rows' split; Y as defined in Sec. II-B). The flat kernel runs when
every hub row has at most 32 chunks and the launch covers more than two
32-column slices (unrolled for 8, 16 or 32 chunks); otherwise the tree does.
Both add in fixed orders. Every element of Y is compared with the oracle at
the edges of the unroll depths: longest hub rows of exactly 8, 9, 16, 17, 32
and 33 chunks, at 1, 2, 4 and 8 slices.
"""
import numpy as np
import pytest

import graphgen
from gpu_helpers import _plan, _spmm_check

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

H = 512  # the default chunk: deg_bound = W * Z = 16 * 32


@pytest.mark.parametrize("chunks", [8, 9, 16, 17, 32, 33])
def test_hub_rows_of_every_unroll_depth(chunks):
    rng = np.random.default_rng(700 + chunks)
    n = 3000
    deg = rng.integers(0, 40, size=n)
    hubs = rng.choice(n, size=12, replace=False)
    deg[hubs] = rng.integers(H + 1, chunks * H + 1, size=12)
    deg[hubs[0]] = chunks * H  # the longest row: exactly `chunks` chunks
    g = graphgen.random_csr(n, chunks * H + 100, deg, seed=800 + chunks)
    p = _plan(g)
    assert p.stats.n_hub_rows == 12
    assert p.stats.max_deg == chunks * H
    for F in (32, 64, 128, 256):  # 1, 2, 4 and 8 slices
        _spmm_check(p, g, F, seed=F)
    p.destroy()
