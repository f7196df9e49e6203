"""The binding refuses operands that do not match the context before any call into the library
(CPU tensors stand in for GPU ones here: shape and type are checked before the device)."""
import pytest
import torch

from paper_2609_19758_amd import fpsketch as fk

N1, N2, N3 = 6, 4, 5


def ops(**kw):
    fk.check_operands(N1, N2, N3, kw.pop("fmt", "bf16"), kw.pop("b_layout", 0), 0, **kw)


def test_wrong_shapes_rejected():
    with pytest.raises(ValueError, match="A: shape"):
        ops(A=torch.zeros(N1, N2 + 1, dtype=torch.bfloat16))
    with pytest.raises(ValueError, match="B: shape"):
        ops(B=torch.zeros(N3, N2, dtype=torch.bfloat16))
    with pytest.raises(ValueError, match="W = B\\^T: shape"):
        ops(B=torch.zeros(N2, N3, dtype=torch.bfloat16), b_layout=1)
    with pytest.raises(ValueError, match="C: shape"):
        ops(C=torch.zeros(N1 * N3 - 1, dtype=torch.float32))
    with pytest.raises(ValueError, match="C: shape"):
        ops(C=torch.zeros(N3, N1, dtype=torch.float32))


def test_wrong_formats_rejected():
    with pytest.raises(ValueError, match="A: dtype"):
        ops(A=torch.zeros(N1, N2, dtype=torch.float16))                  # FP16 into a BF16 ctx
    with pytest.raises(ValueError, match="B: dtype"):
        ops(B=torch.zeros(N2, N3, dtype=torch.bfloat16), fmt="fp16")
    with pytest.raises(ValueError, match="A: dtype"):
        ops(A=torch.zeros(N1, N2, dtype=torch.float32))
    with pytest.raises(ValueError, match="C: dtype"):
        ops(C=torch.zeros(N1, N3, dtype=torch.bfloat16), c_float=True)
    with pytest.raises(ValueError, match="d_dirty"):
        ops(d_dirty=torch.zeros(1, dtype=torch.int64))
    with pytest.raises(ValueError, match="d_dirty"):
        ops(d_dirty=torch.zeros(0, dtype=torch.int32))


def test_layout_and_device_rejected():
    with pytest.raises(ValueError, match="not contiguous"):
        ops(A=torch.zeros(N2, N1, dtype=torch.bfloat16).t())
    with pytest.raises(ValueError, match="expected a GPU tensor"):
        ops(A=torch.zeros(N1, N2, dtype=torch.bfloat16))
    with pytest.raises(ValueError, match="expected a GPU tensor"):
        ops(C=torch.zeros(N1, N3, dtype=torch.float32))
    with pytest.raises(ValueError, match="expected a GPU tensor"):
        ops(d_dirty=torch.zeros(1, dtype=torch.int32))


def test_flat_buffers_of_the_right_size_and_raw_pointers_pass_to_the_device_check():
    # a 1-D tensor with the right element count is accepted up to the device check
    with pytest.raises(ValueError, match="expected a GPU tensor"):
        ops(A=torch.zeros(N1 * N2, dtype=torch.bfloat16))
    # raw integer device pointers and absent arguments are the caller's responsibility
    ops(A=12345, B=None, C=67890, d_dirty=None)
