"""Layout fingerprint pins of the oracle (CPU only).

The paper located a W2 row-order fault by fingerprinting output columns and
printed the 16-row block mapping it found inside each 128-wide N tile,
together with the inverse it applied at load time (Correctness recovery / W2
permutation; tests/golden/w2_row_block_permutation.txt). With
column-fingerprint weights (tests/layout_fingerprint.py) the oracle's
partials name, column by column, the W2 row they came from: the logical
layout decodes to the identity, the paper's mapping planted in the stored W2
decodes to exactly the printed mapping, and the printed inverse restores the
identity.
"""
import os

import numpy as np
import pytest

from oracle import moe
from tests import layout_fingerprint as fp
from tests.conftest import GOLDEN

FAST_TO_REF, INVERSE = fp.read_golden_maps(os.path.join(GOLDEN, "w2_row_block_permutation.txt"))


def _partials(w, H, T=2, fmt="e4m3"):
    r = moe.layer(fp.x_bits(T, H), *w, k=1, logits=np.zeros((T, 1), np.float32), fmt=fmt,
                  keep=True)
    return r["p_slots"][:, 0, :]


def test_printed_maps_are_mutual_inverses():
    assert sorted(FAST_TO_REF) == list(range(8)) and sorted(INVERSE) == list(range(8))
    assert [FAST_TO_REF[INVERSE[j]] for j in range(8)] == list(range(8))
    assert [INVERSE[FAST_TO_REF[j]] for j in range(8)] == list(range(8))


@pytest.mark.parametrize("fmt", ["e4m3", "e2m1", "bf16", None])
@pytest.mark.parametrize("H,I", [(256, 128), (512, 512), (768, 128)])
def test_logical_layout_decodes_to_identity(H, I, fmt):
    p = _partials(fp.weights(H, I), H, fmt=fmt)
    for row in p:
        assert fp.decode(row, H).tolist() == list(range(H))


def test_planted_paper_permutation_is_read_back_and_undone():
    H, I = 512, 128
    w13, w13s, w2, w2s = fp.weights(H, I)
    sw2, sw2s = fp.permute_w2_blocks(w2[0], w2s[0], FAST_TO_REF)
    p = _partials((w13, w13s, sw2[None], sw2s[None]), H)
    maps = fp.block_map(fp.decode(p[0], H))
    assert maps == [FAST_TO_REF] * (H // 128)
    # the inverse applied to the stored rows at load time restores the order
    fw2, fw2s = fp.permute_w2_blocks(sw2, sw2s, INVERSE)
    assert np.array_equal(fw2, w2[0]) and np.array_equal(fw2s, w2s[0])
    p = _partials((w13, w13s, fw2[None], fw2s[None]), H)
    assert fp.decode(p[0], H).tolist() == list(range(H))


def test_every_column_fingerprint_is_distinct_and_exact_in_fp32():
    H = 4096
    p = _partials(fp.weights(H, 128), H, T=1)[0]
    assert np.array_equal(p.astype(np.float32).astype(np.float64), p)
    assert len(set(p.tolist())) == H
    assert fp.decode(p, H).tolist() == list(range(H))
