"""The Python binding's argument checks, without a GPU: every buffer the caller
passes is checked for dtype, contiguity, size and place before its address can
reach the library, and a mis-sized AAD is rejected instead of truncated."""
import numpy as np
import pytest
import torch

import paper_2410_15240_amd as F

KEY, IV = bytes(32), bytes(12)


def u8(n):
    return torch.zeros(n, dtype=torch.uint8)


def test_buffer_check_order_and_messages():
    with pytest.raises(ValueError, match="torch tensor"):
        F._u8(np.zeros(4, np.uint8), "x")
    with pytest.raises(ValueError, match="uint8"):
        F._u8(torch.zeros(4, dtype=torch.int32), "x")
    with pytest.raises(ValueError, match="contiguous"):
        F._u8(u8(8)[::2], "x")
    with pytest.raises(ValueError, match="exactly 5"):
        F._u8(u8(4), "x", numel=5)
    with pytest.raises(ValueError, match="at least 5"):
        F._u8(u8(4), "x", min_numel=5)
    with pytest.raises(ValueError, match="CUDA tensor"):
        F._u8(u8(4), "x", numel=4)
    with pytest.raises(ValueError, match="pinned"):
        F._u8(u8(4), "x", cuda=False, pinned=True)
    assert F._u8(u8(4), "x", numel=4, cuda=False) is not None


@pytest.mark.parametrize("numel,n", [(33, 2), (10, 3), (1, 2), (5, 0)])
def test_aad_that_is_not_n_times_aad_bytes_is_rejected(numel, n):
    with pytest.raises(ValueError):
        F._aad_bytes(u8(numel), n, cuda=False)


def test_aad_bytes_from_shape_or_size():
    assert F._aad_bytes(None, 7) == 0
    assert F._aad_bytes(u8(64), 2, cuda=False) == 32
    assert F._aad_bytes(torch.zeros((3, 1), dtype=torch.uint8), 3, cuda=False) == 1
    assert F._aad_bytes(u8(0), 0, cuda=False) == 0
    assert F._aad_bytes(u8(96), 4, aad_bytes=24, cuda=False) == 24
    with pytest.raises(ValueError):
        F._aad_bytes(u8(96), 4, aad_bytes=32, cuda=False)   # explicit size that does not match
    with pytest.raises(ValueError):
        F._aad_bytes(None, 4, aad_bytes=32)


@pytest.mark.parametrize("call", [
    lambda: F.decrypt_verify(KEY, IV, 4096, u8(8192), u8(32)),
    lambda: F.encrypt_tag(KEY, IV, 4096, u8(8192)),
    lambda: F.decrypt_eager(KEY, IV, 4096, u8(8192), u8(32)),
    lambda: F.apply_verify(KEY, IV, 4096, u8(8192), u8(8192), u8(32)),
    lambda: F.decrypt_verify_ragged(KEY, IV, [0], [16], u8(16), u8(16)),
    lambda: F.encrypt_tag_ragged(KEY, IV, [0], [16], u8(16)),
    lambda: F.pipeline_d2h(KEY, IV, 4096, u8(8192)),
])
def test_host_tensors_are_not_device_buffers(call):
    with pytest.raises(ValueError, match="CUDA tensor"):
        call()


def test_pipeline_needs_pinned_host_ciphertext():
    with pytest.raises(ValueError, match="pinned"):
        F.pipeline_h2d(KEY, IV, 4096, u8(8192), u8(32))


def test_ragged_layout_must_fit_the_buffer():
    with pytest.raises(ValueError, match="past the end"):
        F._ragged_layout([0, 16], [16, 17], 32, "ct")
    with pytest.raises(ValueError, match="differ in length"):
        F._ragged_layout([0, 16], [16], 32, "ct")
    off, ln = F._ragged_layout([0, 16], [16, 16], 32, "ct")
    assert off.dtype == np.uint64 and ln.tolist() == [16, 16]
