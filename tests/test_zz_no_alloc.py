"""dge_score_noalloc through the C ABI (GPU): the scoring entry point that allocates
nothing, against dge_score with a caller workspace and against the oracle, on two calls
in a row whose second is smaller than the first (the shared scratch keeps the first
call's contents), and an oversize geometry refused before any launch."""
import ctypes

import numpy as np
import pytest
import torch

import dge_inputs as di
import oracle
import paper_2609_33334_amd as dge
from paper_2609_33334_amd import _lib

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits)).view(torch.int16).view(torch.bfloat16).to(DEV)


def _case(lens):
    wl = di.small_variant("c2", lens)
    x = di.make_layer(wl, with_v=False)
    g = dge.Geometry(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.window, wl.k_draft,
                     wl.cached_lens, device=DEV)
    return wl, x, g


def test_score_noalloc_matches_score_and_oracle_on_two_calls():
    # the first call is the larger one: the second must not see its leftovers
    for lens in ((2500, 700, 1900, 64), (300, 90)):
        wl, x, g = _case(lens)
        print(f"noalloc score lens={lens}", flush=True)
        q, k = _dev(x.q_bits), _dev(x.k_bits)
        got = dge.score_noalloc(g, dge.ROWS_WINDOW_DRAFT, q, k)
        torch.cuda.synchronize()
        ref = dge.score(g, dge.ROWS_WINDOW_DRAFT, q, k)
        torch.cuda.synchronize()
        assert torch.equal(got.view(torch.int32), ref.view(torch.int32)), lens
        want = oracle.window_scores(x.q, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads,
                                    wl.window, wl.k_draft)
        err = np.abs(got.cpu().numpy().astype(np.float64) - want)
        assert (err <= 1e-3 * np.abs(want) + 1e-20).all(), (lens, float(err.max()))


def test_score_noalloc_other_rows_modes_and_oversize():
    wl, x, g = _case((1200,))
    q, k = _dev(x.q_bits), _dev(x.k_bits)
    nr = wl.window + wl.k_draft
    for mode, sl in ((dge.ROWS_DRAFT, slice(wl.window, nr)), (dge.ROWS_WINDOW, slice(0, wl.window))):
        qm = q[:, sl].contiguous()
        got = dge.score_noalloc(g, mode, qm, k)
        ref = dge.score(g, mode, qm, k)
        torch.cuda.synchronize()
        assert torch.equal(got.view(torch.int32), ref.view(torch.int32)), mode
    # 128 Llama-3-8B layers x 8 sequences of 32K rows (64 such layers fit the scratch)
    big = dge.Geometry(4096, 1024, 128, 32, 2, [32768] * 8, device=DEV)
    assert dge.workspace_size(big, dge.OP_SCORE) > _lib.NOALLOC_SCRATCH_BYTES
    raw = torch.empty(4, dtype=torch.float32, device=DEV)
    st = _lib.lib().dge_score_noalloc(ctypes.byref(big.c), dge.ROWS_WINDOW_DRAFT, q.data_ptr(), k.data_ptr(),
                                      raw.data_ptr(), None)
    assert st == _lib.DGE_ERR_WORKSPACE
