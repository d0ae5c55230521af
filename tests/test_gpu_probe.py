"""The read-only stream probe (profk_debug_read_probe) reads every 16-byte
vector of its buffer exactly once: the XOR of its per-workgroup folds equals
the XOR of all the buffer's words, for every launch shape it accepts."""

import numpy as np
import pytest

import paper_2608_12573_amd as pk
from gpu_util import note, torch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("words", [4, 4 * 1000 + 4, 2**24 + 4 * 77, 2**26])
@pytest.mark.parametrize("per_cu,loads", [(1, 4), (2, 4), (4, 8), (8, 8)])
def test_read_probe_folds_every_word(words, per_cu, loads):
    t = torch()
    host = np.random.default_rng(words + per_cu).integers(0, 2**32, words, dtype=np.uint64).astype(np.uint32)
    g = t.from_numpy(host.view(np.int32)).cuda()
    note(f"read_probe words={words} per_cu={per_cu} loads={loads}")
    out, grid = pk.debug_read_probe(g, per_cu, loads)
    t.cuda.synchronize()
    assert 1 <= grid <= 1024
    folds = out[:grid].cpu().numpy().view(np.uint32)
    assert np.bitwise_xor.reduce(folds) == np.bitwise_xor.reduce(host)
