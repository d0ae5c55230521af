"""The Python binding refuses unusable tensors before anything reaches the
library: wrong rank, dtype or memory layout, host tensors, and caller-given
outputs, workspaces or report buffers that are too small or on the wrong
device.  Every case here is host-only (no GPU), so each error must be raised
before a launch could happen."""

import pytest
import torch

import paper_2608_12573_amd as pk


def _raises(fn, match):
    with pytest.raises(pk.ProfkError, match=match):
        fn()


def test_topk_rejects_host_tensor():
    _raises(lambda: pk.topk(torch.zeros(100), 5), "CUDA tensor")
    _raises(lambda: pk.topk_noalloc(torch.zeros(100), 5), "CUDA tensor")
    _raises(lambda: pk.topk_tau(torch.zeros(100), 5, 0, pk.plan(100, 5)), "CUDA tensor")
    _raises(lambda: pk.debug_filter(torch.zeros(100), 0, pk.plan(100, 5)), "CUDA tensor")


def test_topk_rejects_strided_view():
    # x[::2] would otherwise be read as numel contiguous elements
    _raises(lambda: pk.topk(torch.zeros(200)[::2], 5), "contiguous")
    _raises(lambda: pk.topk_noalloc(torch.zeros(200)[::2], 5), "contiguous")


def test_rank_and_dtype():
    _raises(lambda: pk.topk(torch.zeros(4, 25), 5), "1 dimension")
    _raises(lambda: pk.topk(torch.zeros(100, dtype=torch.float16), 5), "unsupported dtype")
    _raises(lambda: pk.topk(torch.zeros(100, dtype=torch.int32), 5), "unsupported dtype")
    _raises(lambda: pk.topk_rows(torch.zeros(100), 5), "2 dimension")
    _raises(lambda: pk.batchtopk(torch.zeros(100), 5), "2 dimension")


def test_topk_simple_is_fp32_only():
    # a bf16 tensor would be read as 4N bytes from a 2N-byte buffer
    _raises(lambda: pk.topk_simple(torch.zeros(100, dtype=torch.bfloat16), 5), "float32")
    _raises(lambda: pk.topk_simple(torch.zeros(100), 5), "CUDA tensor")
    _raises(lambda: pk.topk_simple(torch.zeros(200)[::2], 5), "contiguous")


def test_rows_layout():
    x = torch.zeros(8, 64)
    _raises(lambda: pk.topk_rows(x.t(), 4), "unit column stride")
    _raises(lambda: pk.topk_rows(x[:, ::2], 4), "unit column stride")
    _raises(lambda: pk.topk_rows(x, 4), "CUDA tensor")
    # strided rows of a wider matrix are fine up to the device check
    _raises(lambda: pk.topk_rows(torch.zeros(8, 100)[:, :64], 4), "CUDA tensor")


def test_batchtopk_needs_contiguous():
    _raises(lambda: pk.batchtopk(torch.zeros(8, 100)[:, :64], 4), "contiguous")
    _raises(lambda: pk.batchtopk(torch.zeros(8, 64), 4), "CUDA tensor")


def test_output_checks_precede_launch():
    """Checked by calling the output helpers on host tensors: wrong dtype,
    too few elements and non-contiguous outputs are refused."""
    x = torch.zeros(100)
    _raises(lambda: pk._buffer(torch.zeros(3), "out[0]", torch.float32, 5, None), "at least 5")
    _raises(lambda: pk._buffer(torch.zeros(5, dtype=torch.int32), "out[1]", torch.int64, 5, None), "int64")
    _raises(lambda: pk._buffer(torch.zeros(10)[::2], "out[0]", torch.float32, 5, None), "contiguous")
    _raises(lambda: pk._bytes_buffer(torch.zeros(2, dtype=torch.uint8), "info", pk.INFO_BYTES, None), "bytes")
    _raises(lambda: pk._buffer(torch.zeros(5), "out[0]", torch.float32, 5, x.device), "CUDA tensor")


def test_workspace_size_counts_bytes():
    """A workspace tensor of any dtype is measured in bytes."""
    p = pk.plan(2**20, 64)
    need = pk.workspace_size(p, pk.F32)
    _raises(lambda: pk._bytes_buffer(torch.zeros(need // 4 - 1, dtype=torch.float32), "ws", need, None), "bytes")
    # big enough in bytes: only the device check is left
    _raises(lambda: pk._bytes_buffer(torch.zeros(need // 4 + 1, dtype=torch.float32), "ws", need, None),
            "CUDA tensor")


def test_sae_inputs():
    bf = torch.bfloat16
    x, w, b = torch.zeros(4, 64, dtype=bf), torch.zeros(16, 64, dtype=bf), torch.zeros(16)
    _raises(lambda: pk.sae_encode_topk(x, w, b, 2), "CUDA tensor")
    _raises(lambda: pk.sae_encode_dense(x.float(), w, b), "bfloat16")
    _raises(lambda: pk.sae_encode_dense(x, w, b), "CUDA tensor")
    _raises(lambda: pk.sae_decode(torch.zeros(8), torch.zeros(8, dtype=torch.int64), w, torch.zeros(64), 4),
            "CUDA tensor")
