"""Argument checks of the Python binding (CPU only, nothing is launched).

The C ABI receives raw pointers, so the binding refuses tensors whose element type,
size or device the library would misread: an fp16 tensor read as float32, int64
positions read as pairs of int32, or a host pointer handed to a kernel."""
import pytest
import torch

import paper_2609_33334_amd as dge


def test_rope_refuses_fp16_rows():
    x = torch.zeros(2, 8, 128, dtype=torch.float16)
    with pytest.raises(TypeError, match="bfloat16 or float32"):
        dge.rope(x, torch.arange(8, dtype=torch.int32))


def test_rope_refuses_int64_positions():
    x = torch.zeros(2, 8, 128, dtype=torch.bfloat16)
    with pytest.raises(TypeError, match="int32"):
        dge.rope(x, torch.arange(8))


def test_rope_refuses_short_positions_and_host_tensors():
    x = torch.zeros(2, 8, 128, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="at least 8"):
        dge.rope(x, torch.arange(5, dtype=torch.int32))
    with pytest.raises(ValueError, match="needs a GPU tensor"):
        dge.rope(x, torch.arange(8, dtype=torch.int32))


def test_score_refuses_wrong_dtype_size_and_device():
    g = dge.Geometry(4, 2, 64, 2, 1, [40, 50], dtype=dge.DGE_BF16, device="cpu")
    q = torch.zeros(4, 2 * 3, 64, dtype=torch.bfloat16)
    k = torch.zeros(2, 90, 64, dtype=torch.bfloat16)
    raw = torch.zeros(2, 90, dtype=torch.float32)
    with pytest.raises(TypeError, match="dtype"):
        dge.score(g, dge.ROWS_WINDOW_DRAFT, q.float(), k, raw=raw)
    with pytest.raises(ValueError, match="elements"):
        dge.score(g, dge.ROWS_WINDOW_DRAFT, q, k[:, :60].contiguous(), raw=raw)
    with pytest.raises(ValueError, match="needs a GPU tensor"):
        dge.score(g, dge.ROWS_WINDOW_DRAFT, q, k, raw=raw)


def test_select_and_compact_refuse_wrong_index_types():
    g = dge.Geometry(4, 2, 64, 2, 1, [40, 50], dtype=dge.DGE_F32, device="cpu")
    scores = torch.zeros(2, 90, dtype=torch.float32)
    with pytest.raises(TypeError, match="dtype"):
        dge.select_topb(g, scores.double(), 1, 3, 4, idx=torch.zeros(2, 2, 4, dtype=torch.int32),
                        n_kept=torch.zeros(2, dtype=torch.int32))
    k = torch.zeros(2, 90, 64)
    with pytest.raises(TypeError, match="dtype"):
        dge.compact(g, torch.zeros(2, 2, 4, dtype=torch.int64), torch.zeros(2, dtype=torch.int32),
                    4, 3, k, k, k_out=torch.zeros(2, 2, 7, 64), v_out=torch.zeros(2, 2, 7, 64))
