"""CPU checks of the C ABI: the library loads, exports every symbol include/dge.h
declares, and rejects bad arguments on the host before launching anything.
No call here reaches the GPU (every call either fails validation or is host-only)."""
import ctypes
import json
import os
import re

import numpy as np
import pytest

import oracle
from paper_2609_33334_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dge.h")


@pytest.fixture(scope="module")
def L():
    return _lib.lib()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dge_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol(L):
    names = _declared_functions()
    assert set(names) == set(_lib.EXPORTS), names
    for n in names:
        assert hasattr(L, n), n


def test_abi_version_and_status_strings(L):
    assert L.dge_abi_version() == _lib.ABI_VERSION
    for s in range(5):
        assert _lib.status_string(s).startswith(["DGE_OK", "DGE_ERR_INVALID", "DGE_ERR_UNSUPPORTED",
                                                 "DGE_ERR_WORKSPACE", "DGE_ERR_HIP"][s])
    assert "unknown" in _lib.status_string(99)


def test_geom_struct_layout_matches_c():
    # int32 x6 | ptr | ptr | int64 | int32 (+pad): offsets per the C layout rules
    G = _lib.Geom
    assert G.kv_offsets.offset == 24 and G.kv_offsets_host.offset == 32
    assert G.kv_head_stride.offset == 40 and G.dtype.offset == 48
    assert ctypes.sizeof(G) == 56


def test_pyramid_budgets_host_matches_paper_examples(L):
    cases = json.load(open(os.path.join(ROOT, "tests", "golden", "pyramidkv_worked_examples.json")))["cases"]
    for c in cases:
        out = (ctypes.c_int32 * c["n_layers"])()
        assert L.dge_pyramid_budgets(c["B"], c["w"], c["n_layers"], 20, out) == 0
        past = np.array(list(out)) - c["w"]
        if "last_layers_past" in c:
            assert past[-len(c["last_layers_past"]):].tolist() == c["last_layers_past"]
        if "every_layer_past" in c:
            assert (past == c["every_layer_past"]).all()
        assert np.array_equal(np.array(list(out)), oracle.pyramid_budgets(c["B"], c["w"], c["n_layers"]))
    for B, w, n in [(2048, 32, 32), (128, 8, 32), (64, 8, 1), (8, 8, 5)]:
        out = (ctypes.c_int32 * n)()
        assert L.dge_pyramid_budgets(B, w, n, 20, out) == 0
        assert list(out) == oracle.pyramid_budgets(B, w, n).tolist()


def test_pyramid_budgets_rejects(L):
    out = (ctypes.c_int32 * 4)()
    assert L.dge_pyramid_budgets(4, 8, 4, 20, out) == _lib.DGE_ERR_INVALID      # B < w
    assert L.dge_pyramid_budgets(64, 8, 0, 20, out) == _lib.DGE_ERR_INVALID
    assert L.dge_pyramid_budgets(64, 8, 4, 0, out) == _lib.DGE_ERR_INVALID
    assert L.dge_pyramid_budgets(64, 8, 4, 20, None) == _lib.DGE_ERR_INVALID


# ------------------------------------------------------------------------------------------
# Host validation: every call below must fail before any launch.
# Device pointers are fake (aligned, never dereferenced on the host).
# ------------------------------------------------------------------------------------------
FAKE = 1 << 32          # 16-byte aligned fake device address


class _G:
    def __init__(self, lens=(100, 60), hq=8, hkv=2, d=128, w=8, k=2, dtype=0, stride=None):
        self.offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
        T = int(self.offs[-1])
        self.g = _lib.Geom(len(lens), hq, hkv, d, w, k, FAKE, self.offs.ctypes.data,
                           T * d if stride is None else stride, dtype)

    @property
    def p(self):
        return ctypes.byref(self.g)


def _score(L, G, rows=0, q=FAKE, k=FAKE, raw=FAKE, ws=FAKE, nbytes=1 << 40):
    return L.dge_score(G.p, rows, q, k, raw, ws, nbytes, None)


def test_score_validation(L):
    assert _score(L, _G(hq=6, hkv=4)) == _lib.DGE_ERR_INVALID          # H_q % H_kv
    assert _score(L, _G(d=96)) == _lib.DGE_ERR_UNSUPPORTED              # head_dim
    assert _score(L, _G(lens=(100, 9))) == _lib.DGE_ERR_INVALID          # N_b < w + k
    assert _score(L, _G(w=0, k=0)) == _lib.DGE_ERR_INVALID               # no scoring rows
    assert _score(L, _G(k=0), rows=_lib.ROWS_DRAFT) == _lib.DGE_ERR_INVALID
    assert _score(L, _G(), rows=3) == _lib.DGE_ERR_INVALID
    assert _score(L, _G(), q=FAKE + 4) == _lib.DGE_ERR_INVALID           # misaligned
    assert _score(L, _G(), raw=None) == _lib.DGE_ERR_INVALID
    assert _score(L, _G(), ws=None) == _lib.DGE_ERR_WORKSPACE
    assert _score(L, _G(), nbytes=16) == _lib.DGE_ERR_WORKSPACE
    assert _score(L, _G(dtype=5)) == _lib.DGE_ERR_INVALID
    assert _score(L, _G(stride=10)) == _lib.DGE_ERR_INVALID              # stride < T*d
    g = _G()
    g.offs[0] = 1
    assert _score(L, g) == _lib.DGE_ERR_INVALID                          # offsets[0] != 0
    g = _G(lens=(50, 50))
    g.offs[1], g.offs[2] = 80, 70
    assert _score(L, g) == _lib.DGE_ERR_INVALID                          # decreasing offsets
    assert L.dge_score(None, 0, FAKE, FAKE, FAKE, FAKE, 1 << 40, None) == _lib.DGE_ERR_INVALID
    assert L.dge_score_lse(_G().p, 0, FAKE, FAKE, None, FAKE, None) == _lib.DGE_ERR_INVALID
    assert L.dge_score_lse(_G(d=96).p, 0, FAKE, FAKE, FAKE, FAKE, None) == _lib.DGE_ERR_UNSUPPORTED
    assert L.dge_score_lse(_G(lens=(100, 9)).p, 0, FAKE, FAKE, FAKE, FAKE, None) == _lib.DGE_ERR_INVALID


def test_score_noalloc_validation(L):
    """dge_score_noalloc: dge_score's checks, and a geometry whose partials exceed the fixed
    scratch is refused (DGE_ERR_WORKSPACE) before the scratch address is even looked up."""
    def call(G, rows=0, q=FAKE, k=FAKE, raw=FAKE):
        return L.dge_score_noalloc(G.p, rows, q, k, raw, None)
    assert call(_G(hq=6, hkv=4)) == _lib.DGE_ERR_INVALID
    assert call(_G(d=96)) == _lib.DGE_ERR_UNSUPPORTED
    assert call(_G(lens=(100, 9))) == _lib.DGE_ERR_INVALID
    assert call(_G(w=0, k=0)) == _lib.DGE_ERR_INVALID
    assert call(_G(), raw=None) == _lib.DGE_ERR_INVALID
    assert call(_G(), k=FAKE + 8) == _lib.DGE_ERR_INVALID
    # 8 sequences of 32K rows over 1024 KV heads (128 Llama-3-8B layers), 136 query rows
    # per head: ~23.6 MB of partials
    big = _G(lens=(32768,) * 8, hq=4096, hkv=1024, w=32, k=2)
    n = ctypes.c_size_t(0)
    assert L.dge_workspace_size(big.p, 0, ctypes.byref(n)) == 0
    assert n.value > _lib.NOALLOC_SCRATCH_BYTES
    assert call(big) == _lib.DGE_ERR_WORKSPACE
    assert L.dge_score_noalloc(None, 0, FAKE, FAKE, FAKE, None) == _lib.DGE_ERR_INVALID


def test_score_with_lse_and_evicted_mass_validation(L):
    G = _G()
    def sl(g=G, lse=FAKE, ws=FAKE, nbytes=1 << 40):
        return L.dge_score_with_lse(g.p, 0, FAKE, FAKE, FAKE, lse, ws, nbytes, None)
    assert sl(lse=None) == _lib.DGE_ERR_INVALID
    assert sl(lse=FAKE + 4) == _lib.DGE_ERR_INVALID
    assert sl(ws=None) == _lib.DGE_ERR_WORKSPACE
    assert sl(g=_G(d=96)) == _lib.DGE_ERR_UNSUPPORTED

    def em(g=G, n_q=10, q_from_end=10, n_select=20, n_tail=10, rho=FAKE, lse=FAKE):
        return L.dge_evicted_mass(g.p, FAKE, n_q, q_from_end, FAKE, n_select, n_tail, FAKE, lse,
                                  rho, FAKE, FAKE, None)
    assert em(n_q=0) == _lib.DGE_ERR_INVALID
    assert em(q_from_end=11) == _lib.DGE_ERR_INVALID         # rows beyond the tail
    assert em(n_q=11, q_from_end=10, n_tail=12) == _lib.DGE_ERR_INVALID   # rows past the cache end
    assert em(n_tail=0, q_from_end=0) == _lib.DGE_ERR_INVALID
    assert em(n_select=-1) == _lib.DGE_ERR_INVALID
    assert em(rho=None) == _lib.DGE_ERR_INVALID
    assert em(lse=FAKE + 2) == _lib.DGE_ERR_INVALID
    assert em(g=_G(hq=18, hkv=1)) == _lib.DGE_ERR_UNSUPPORTED    # more than 8 heads per group


def test_project_rope_validation(L):
    n = ctypes.c_size_t(0)
    assert L.dge_project_rope_workspace(34, 4096, 32, 128, ctypes.byref(n)) == 0 and n.value > 0
    need = n.value
    assert L.dge_project_rope_workspace(8194, 4096, 32, 128, ctypes.byref(n)) == 0 and n.value == 0
    assert L.dge_project_rope_workspace(34, 4096, 32, 96, ctypes.byref(n)) == _lib.DGE_ERR_UNSUPPORTED
    assert L.dge_project_rope_workspace(34, 4000, 32, 128, ctypes.byref(n)) == _lib.DGE_ERR_UNSUPPORTED
    assert L.dge_project_rope_workspace(34, 4096, 32, 128, None) == _lib.DGE_ERR_INVALID
    def call(rows=34, hidden=4096, heads=32, d=128, theta=5e5, ws=FAKE, nbytes=1 << 40, x=FAKE):
        return L.dge_project_rope(rows, hidden, x, heads, d, FAKE, FAKE, theta, FAKE, ws, nbytes, None)
    assert call(ws=None) == _lib.DGE_ERR_WORKSPACE
    assert call(nbytes=need - 1) == _lib.DGE_ERR_WORKSPACE
    assert call(theta=1.0) == _lib.DGE_ERR_INVALID
    assert call(rows=-1) == _lib.DGE_ERR_INVALID
    assert call(x=FAKE + 2) == _lib.DGE_ERR_INVALID
    assert call(d=96) == _lib.DGE_ERR_UNSUPPORTED
    assert call(rows=0, ws=None) == _lib.DGE_OK            # nothing to do, nothing launched


def test_workspace_size(L):
    g = _G()
    n = ctypes.c_size_t(0)
    for op in (0, 1, 2):
        assert L.dge_workspace_size(g.p, op, ctypes.byref(n)) == 0 and n.value > 0
    assert L.dge_workspace_size(g.p, 7, ctypes.byref(n)) == _lib.DGE_ERR_INVALID
    assert L.dge_workspace_size(g.p, 0, None) == _lib.DGE_ERR_INVALID


def test_select_validation(L):
    g = _G()
    def sel(pool=7, n_tail=10, n_select=20, idx=FAKE, nk=FAKE, ws=FAKE, nbytes=1 << 40):
        return L.dge_select_topb(g.p, FAKE, pool, n_tail, n_select, idx, nk, ws, nbytes, None)
    assert sel(pool=6) == _lib.DGE_ERR_INVALID
    assert sel(pool=0) == _lib.DGE_ERR_INVALID
    assert sel(n_select=-1) == _lib.DGE_ERR_INVALID
    assert sel(n_tail=61) == _lib.DGE_ERR_INVALID          # > N_b of the second sequence
    assert sel(n_tail=-1) == _lib.DGE_ERR_INVALID
    assert sel(idx=None) == _lib.DGE_ERR_INVALID
    assert sel(ws=None) == _lib.DGE_ERR_WORKSPACE
    assert sel(nbytes=8) == _lib.DGE_ERR_WORKSPACE


def test_streaming_compact_h2o_validation(L):
    g = _G()
    assert L.dge_select_streaming(g.p, -1, 10, FAKE, FAKE, None) == _lib.DGE_ERR_INVALID
    assert L.dge_select_streaming(g.p, 4, 61, FAKE, FAKE, None) == _lib.DGE_ERR_INVALID
    assert L.dge_compact(g.p, FAKE, FAKE, -1, 10, FAKE, FAKE, FAKE, FAKE, None) == _lib.DGE_ERR_INVALID
    assert L.dge_compact(g.p, FAKE, FAKE, 5, 61, FAKE, FAKE, FAKE, FAKE, None) == _lib.DGE_ERR_INVALID
    assert L.dge_compact(g.p, FAKE, FAKE, 5, 10, FAKE, FAKE, FAKE + 8, FAKE, None) == _lib.DGE_ERR_INVALID
    assert L.dge_h2o_colsum(_G(dtype=1).p, FAKE, FAKE, None, FAKE, FAKE, 1 << 40, None) == _lib.DGE_ERR_UNSUPPORTED
    assert L.dge_h2o_colsum(_G(d=64).p, FAKE, FAKE, None, FAKE, FAKE, 1 << 40, None) == _lib.DGE_ERR_UNSUPPORTED
    assert L.dge_h2o_colsum(g.p, FAKE, FAKE, None, FAKE, None, 0, None) == _lib.DGE_ERR_WORKSPACE
    assert L.dge_h2o_colsum(g.p, FAKE, FAKE, FAKE, FAKE, None, 0, None) == _lib.DGE_ERR_WORKSPACE
    assert L.dge_h2o_colsum(_G(hq=16, hkv=2).p, FAKE, FAKE, None, FAKE, FAKE, 1 << 40, None) == _lib.DGE_ERR_UNSUPPORTED


def test_cache_attention_validation(L):
    g = _G()
    def att(geom=g, q=FAKE, n_q=3, q_from_end=0, kc=FAKE, vc=FAKE, n_select=20, n_tail=10,
            nk=FAKE, out=FAKE, lse=FAKE):
        return L.dge_cache_attention(geom.p, q, n_q, q_from_end, kc, vc, n_select, n_tail, nk,
                                     out, lse, None)
    assert att(n_q=0) == _lib.DGE_ERR_INVALID
    assert att(n_select=-1) == _lib.DGE_ERR_INVALID
    assert att(n_tail=-1) == _lib.DGE_ERR_INVALID
    assert att(q_from_end=11) == _lib.DGE_ERR_INVALID        # rows before the tail start
    assert att(n_select=0, n_tail=0, q_from_end=0) == _lib.DGE_ERR_INVALID
    assert att(q=None) == _lib.DGE_ERR_INVALID
    assert att(kc=FAKE + 4) == _lib.DGE_ERR_INVALID
    assert att(lse=FAKE + 2) == _lib.DGE_ERR_INVALID
    assert att(geom=_G(hq=18, hkv=2)) == _lib.DGE_ERR_UNSUPPORTED   # 9 query heads per KV head
    assert att(geom=_G(d=96)) == _lib.DGE_ERR_UNSUPPORTED


def test_retained_runs_validation(L):
    g = _G()
    def runs(geom=g, idx=FAKE, nk=FAKE, n_select=20, out=FAKE, mean=FAKE):
        return L.dge_retained_runs(geom.p, idx, nk, n_select, out, mean, None)
    assert runs(n_select=-1) == _lib.DGE_ERR_INVALID
    assert runs(idx=None) == _lib.DGE_ERR_INVALID
    assert runs(nk=None) == _lib.DGE_ERR_INVALID
    assert runs(out=None) == _lib.DGE_ERR_INVALID
    assert runs(mean=FAKE + 2) == _lib.DGE_ERR_INVALID
    assert runs(idx=FAKE + 1) == _lib.DGE_ERR_INVALID


def test_select_compact_layers_validation(L):
    g = _G()
    ns = (ctypes.c_int32 * 3)(10, 20, 5)
    def call(n_layers=3, arr=ns, pool=7, tail=10, idx=FAKE, ws=FAKE, nbytes=1 << 40, k=FAKE):
        return L.dge_select_compact_layers(g.p, n_layers, FAKE, pool, tail, arr, idx, FAKE, k,
                                           FAKE, FAKE, FAKE, ws, nbytes, None)
    assert call(n_layers=0) == _lib.DGE_ERR_INVALID
    assert call(arr=None) == _lib.DGE_ERR_INVALID
    assert call(arr=(ctypes.c_int32 * 3)(10, -1, 5)) == _lib.DGE_ERR_INVALID
    assert call(pool=4) == _lib.DGE_ERR_INVALID
    assert call(tail=61) == _lib.DGE_ERR_INVALID          # longer than the 60-row sequence
    assert call(idx=None) == _lib.DGE_ERR_INVALID
    assert call(k=FAKE + 8) == _lib.DGE_ERR_INVALID
    assert call(ws=None) == _lib.DGE_ERR_WORKSPACE
    assert call(nbytes=16) == _lib.DGE_ERR_WORKSPACE


def test_compact_inplace_validation(L):
    g = _G()
    def call(n_select=20, n_tail=10, idx=FAKE, nk=FAKE, k=FAKE, v=FAKE + 4096):
        return L.dge_compact_inplace(g.p, idx, nk, n_select, n_tail, k, v, None)
    assert call(n_select=-1) == _lib.DGE_ERR_INVALID
    assert call(n_tail=61) == _lib.DGE_ERR_INVALID
    assert call(v=FAKE) == _lib.DGE_ERR_INVALID            # k and v must be distinct
    assert call(nk=None) == _lib.DGE_ERR_INVALID
    assert call(idx=None) == _lib.DGE_ERR_INVALID
    assert call(k=FAKE + 8) == _lib.DGE_ERR_INVALID


def test_row_counts_bounded(L):
    # n_select + n_tail must stay a valid int32 row count
    g = _G()
    big = 2 ** 31 - 1
    assert L.dge_select_topb(g.p, FAKE, 7, 10, big, FAKE, FAKE, FAKE, 1 << 40, None) == _lib.DGE_ERR_INVALID
    assert L.dge_compact(g.p, FAKE, FAKE, big, 10, FAKE, FAKE, FAKE, FAKE, None) == _lib.DGE_ERR_INVALID
    assert L.dge_compact_inplace(g.p, FAKE, FAKE, big, 10, FAKE, FAKE + 4096, None) == _lib.DGE_ERR_INVALID
    ns = (ctypes.c_int32 * 2)(10, big)
    assert L.dge_select_compact_layers(g.p, 2, FAKE, 7, 10, ns, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                       FAKE, 1 << 40, None) == _lib.DGE_ERR_INVALID


def test_rope_validation(L):
    pos = FAKE
    def call(h=4, n=10, d=128, dt=0, stride=1280, p=pos, theta=500000.0, x=FAKE):
        return L.dge_rope(h, n, d, dt, stride, p, theta, x, None)
    assert call(h=0) == _lib.DGE_ERR_INVALID
    assert call(n=-1) == _lib.DGE_ERR_INVALID
    assert call(d=127) == _lib.DGE_ERR_UNSUPPORTED
    assert call(d=66, stride=660) == _lib.DGE_ERR_UNSUPPORTED      # head_dim not a multiple of 4
    assert call(stride=1281) == _lib.DGE_ERR_INVALID               # heads not 8-byte aligned
    assert call(d=256, stride=2560) == _lib.DGE_ERR_UNSUPPORTED
    assert call(dt=7) == _lib.DGE_ERR_INVALID
    assert call(theta=1.0) == _lib.DGE_ERR_INVALID
    assert call(theta=float("nan")) == _lib.DGE_ERR_INVALID
    assert call(stride=1279) == _lib.DGE_ERR_INVALID
    assert call(p=None) == _lib.DGE_ERR_INVALID
    assert call(x=FAKE + 2) == _lib.DGE_ERR_INVALID
    assert call(n=0, p=None, x=None) == _lib.DGE_OK            # nothing to rotate, nothing launched
