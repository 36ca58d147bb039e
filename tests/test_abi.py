"""C-ABI checks that need no GPU: the library loads, exports every declared entry point, and
rejects bad arguments on the host before any HIP call (only pointers that fail validation are
ever passed, so nothing reaches a device)."""
import ctypes
import os
import re

import pytest
import torch

from paper_2608_01662_amd import lsa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lsa.h")

pytestmark = pytest.mark.skipif(not os.path.exists(lsa.LIB_PATH), reason="liblsa.so not built")

OK, INVALID, UNSUPPORTED, WORKSPACE = 0, 1, 2, 3
FAKE = ctypes.c_void_p(0x100000)       # aligned, never dereferenced: every call below fails validation
MISALIGNED = ctypes.c_void_p(0x100001)


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]*?\b(lsa_\w+)\s*\(", text, re.M)))


def test_exports_every_declared_symbol():
    L = lsa.lib()
    names = declared_functions()
    assert len(names) >= 10, names
    for n in names:
        assert hasattr(L, n), f"{n} declared in lsa.h but not exported"


def test_version_and_status_strings():
    L = lsa.lib()
    assert lsa.version().startswith("lsa-mi355x")
    for code, name in [(0, b"LSA_OK"), (1, b"LSA_ERR_INVALID_ARG"), (2, b"LSA_ERR_UNSUPPORTED"),
                       (3, b"LSA_ERR_WORKSPACE"), (4, b"LSA_ERR_HIP"), (99, b"LSA_ERR_UNKNOWN")]:
        assert L.lsa_status_string(code) == name


def P(**kw):
    base = dict(n_heads=32, head_dim=128, fp8=True, page=128, sub_block=128, keep_pages=64,
                k_sparse=2048, k_sink=4, k_swa=1024, run_align=128)
    base.update(kw)
    return lsa.IndexParams(**base)


def prefill(prm, q_start=0, n_q=16, n_kv=4096, q=FAKE, w=FAKE, k=FAKE, ks=FAKE, bk=FAKE, idx=FAKE, cnt=FAKE,
            runs=None, rc=None, pages=None, ws=FAKE, wsb=1 << 40):
    L = lsa.lib()
    return L.lsa_index_prefill(ctypes.byref(prm.c()), q_start, n_q, n_kv, q, w, k, ks, bk, idx, cnt, runs, rc,
                               pages, ws, wsb, None)


@pytest.mark.parametrize("kw,status", [
    (dict(n_heads=0), UNSUPPORTED), (dict(n_heads=33), UNSUPPORTED), (dict(head_dim=96), UNSUPPORTED),
    (dict(page=48), UNSUPPORTED), (dict(page=512, sub_block=512, k_swa=1024), UNSUPPORTED),
    (dict(sub_block=3), UNSUPPORTED), (dict(page=128, sub_block=2), UNSUPPORTED),
    (dict(k_sparse=0), INVALID), (dict(k_sink=-1), INVALID), (dict(run_align=0), INVALID),
    (dict(keep_pages=8, k_swa=64), UNSUPPORTED),
])
def test_bad_index_params(kw, status):
    assert prefill(P(**kw)) == status
    assert lsa.lib().lsa_index_workspace_size(ctypes.byref(P(**kw).c()), 16, 4096) == 0


def test_unknown_pooling_rejected():
    c = P().c()
    c.pooling = 7
    L = lsa.lib()
    assert L.lsa_index_prefill(ctypes.byref(c), 0, 16, 4096, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None,
                               None, FAKE, 1 << 40, None) == INVALID
    assert L.lsa_block_minmax(ctypes.byref(c), 4096, FAKE, FAKE, FAKE, None) == INVALID


def test_negative_hi_min_kv_rejected():
    c = P().c()
    c.hi_min_kv = -1
    assert lsa.lib().lsa_index_prefill(ctypes.byref(c), 0, 16, 4096, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None,
                                       None, None, FAKE, 1 << 40, None) == INVALID


def test_adaptive_dispatch_workspace():
    """Below the dispatch length the workspace is the flat plan's (no page scores), above it the
    hierarchical one's."""
    L = lsa.lib()
    hi = P(hi_min_kv=0)
    auto = P(hi_min_kv=8192)
    flat = P(keep_pages=0)
    ws = lambda prm, kv: L.lsa_index_workspace_size(ctypes.byref(prm.c()), 64, kv)
    assert ws(auto, 8192) == ws(flat, 8192) != ws(hi, 8192)
    assert ws(auto, 8193) == ws(hi, 8193)


def test_bad_block_cache_arguments():
    """Block-cache calls validate before launching: the rows list of an update must be given and
    8-byte aligned, keys and output 16-byte aligned, a scale exactly for fp8 keys."""
    L = lsa.lib()
    prm = P(pooling="minmax").c()
    assert L.lsa_block_keys_update(ctypes.byref(prm), 4, None, 4096, FAKE, FAKE, FAKE, None) == INVALID
    assert L.lsa_block_keys_update(ctypes.byref(prm), 4, ctypes.c_void_p(0x100004), 4096, FAKE, FAKE, FAKE,
                                   None) == INVALID
    assert L.lsa_block_keys_update(ctypes.byref(prm), 4, FAKE, -1, FAKE, FAKE, FAKE, None) == INVALID
    assert L.lsa_block_minmax(ctypes.byref(prm), 4096, MISALIGNED, FAKE, FAKE, None) == INVALID
    assert L.lsa_block_minmax(ctypes.byref(prm), 4096, FAKE, None, FAKE, None) == INVALID      # fp8 needs scales
    assert L.lsa_block_keys_update(ctypes.byref(prm), 0, None, 4096, None, None, None, None) == OK   # no rows


def test_bad_index_arguments():
    prm = P()
    assert prefill(prm, q_start=4090, n_q=16, n_kv=4096) == INVALID           # rows past the cache
    assert prefill(prm, q_start=(1 << 63) - 8, n_q=16) == INVALID               # no signed overflow in the bound
    assert prefill(prm, n_q=-1) == INVALID
    assert prefill(prm, q=None) == INVALID
    assert prefill(prm, ks=None) == INVALID                                   # fp8 needs scales
    assert prefill(P(fp8=False)) == INVALID                                   # bf16 must not get scales
    assert prefill(prm, bk=None) == INVALID                                   # HI needs mean keys
    assert prefill(prm, runs=FAKE, rc=None) == INVALID
    assert prefill(prm, runs=ctypes.c_void_p(0x100004), rc=FAKE) == INVALID   # runs: 8-byte (start, len) stores
    assert prefill(prm, q=MISALIGNED) == INVALID
    assert prefill(prm, ws=None) == WORKSPACE
    assert prefill(prm, wsb=16) == WORKSPACE
    assert prefill(prm, ws=ctypes.c_void_p(0x100080)) == WORKSPACE             # not 256-byte aligned
    assert prefill(P(keep_pages=0), pages=FAKE) == INVALID                    # pages need HI mode
    # an index list (plus the recalled pages) beyond one workgroup's LDS; long candidate rows
    # alone are fine (their keys stay in global memory)
    assert prefill(P(keep_pages=1024, page=128, k_sparse=30000)) == UNSUPPORTED
    assert b"LDS" in lsa.lib().lsa_last_error()


def test_bad_decode_arguments():
    L = lsa.lib()
    prm = P(page=64, sub_block=64, keep_pages=128, k_swa=256)

    def dec(batch=4, ctx=FAKE, table=FAKE, max_pages=2048, kv_page=64, n_phys=1000, **kw):
        return L.lsa_index_decode(ctypes.byref(prm.c()), batch, ctx, table, max_pages, kv_page, n_phys, FAKE,
                                  FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, None, kw.get("ws", FAKE),
                                  kw.get("wsb", 1 << 40), None)
    assert dec(kv_page=32) == UNSUPPORTED
    assert dec(ctx=None) == INVALID
    assert dec(max_pages=0) == INVALID
    assert dec(batch=-1) == INVALID
    assert dec(wsb=0) == WORKSPACE


def test_static_decode_arguments():
    """lsa_index_decode_static (scratch in the library's fixed array) validates like
    lsa_index_decode and rejects, before any HIP call, a call whose single row needs more
    scratch than the array holds (flat mode over 2^20 pages of 64 tokens: 256 MB per row)."""
    L = lsa.lib()
    hi = P(page=64, sub_block=64, keep_pages=128, k_swa=256)

    def dec(prm=hi, batch=4, ctx=FAKE, table=FAKE, max_pages=2048, kv_page=64, n_phys=1000):
        return L.lsa_index_decode_static(ctypes.byref(prm.c()), batch, ctx, table, max_pages, kv_page, n_phys, FAKE,
                                         FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, None, None)
    assert dec(kv_page=32) == UNSUPPORTED
    assert dec(ctx=None) == INVALID
    assert dec(max_pages=0) == INVALID
    assert dec(batch=-1) == INVALID
    assert dec(prm=P(page=64, sub_block=64, keep_pages=0, k_swa=256), max_pages=1 << 20) == WORKSPACE
    assert b"scratch" in L.lsa_last_error()
    assert dec(batch=0) == OK                                                  # nothing to do, nothing touched


def test_bad_attention_arguments():
    L = lsa.lib()
    mla = lsa.AttnParams(sm_scale=0.07, **lsa.MLA)

    def attn(prm=mla, n_rows=8, q=FAKE, kv=FAKE, v=None, n_kv=100, idx=FAKE, cnt=FAKE, k_cap=64, table=None,
             max_pages=0, kv_page=0, rps=1, out=FAKE, lse=None, ws=FAKE, wsb=1 << 40):
        return L.lsa_sparse_attn(ctypes.byref(prm.c()), n_rows, q, kv, v, n_kv, idx, cnt, k_cap, table, max_pages,
                                 kv_page, rps, out, lse, ws, wsb, None)
    assert attn(prm=lsa.AttnParams(64, 576, 512, False, 0.07)) == UNSUPPORTED
    assert attn(prm=lsa.AttnParams(32, 576, 512, True, 0.07)) == UNSUPPORTED
    assert attn(prm=lsa.AttnParams(64, 576, 512, True, 0.0)) == INVALID
    assert attn(v=FAKE) == INVALID                                             # latent cache takes no V
    assert attn(prm=lsa.AttnParams(sm_scale=0.1, **lsa.MQA)) == INVALID        # MQA needs V
    assert attn(n_kv=0) == INVALID
    assert attn(k_cap=0) == INVALID
    assert attn(out=None) == INVALID
    assert attn(q=MISALIGNED) == INVALID
    assert attn(table=FAKE, max_pages=0) == INVALID
    assert attn(n_rows=8, table=FAKE, max_pages=4, kv_page=64, ws=None) == WORKSPACE


def test_bad_run_form_attention_arguments():
    """lsa_sparse_attn_runs validates on the host before any launch."""
    L = lsa.lib()
    mla = lsa.AttnParams(sm_scale=0.07, **lsa.MLA)
    mqa = lsa.AttnParams(sm_scale=0.1, **lsa.MQA)

    def att(prm=mla, n_rows=8, q=FAKE, kv=FAKE, v=None, n_kv=4096, runs=FAKE, rc=FAKE, k_cap=64, table=None,
            max_pages=0, kv_page=0, rps=1, out=FAKE, lse=None, ws=FAKE, wsb=1 << 40):
        return L.lsa_sparse_attn_runs(ctypes.byref(prm.c()), n_rows, q, kv, v, n_kv, runs, rc, k_cap, table, max_pages,
                                      kv_page, rps, out, lse, ws, wsb, None)
    assert att(prm=mqa) == INVALID                                             # MQA needs v
    assert att(v=FAKE) == INVALID                                              # latent cache takes no v
    assert att(runs=None) == INVALID
    assert att(rc=None) == INVALID
    assert att(runs=ctypes.c_void_p(0x100004)) == INVALID                      # 8-byte (start, len) pairs
    assert att(k_cap=0) == INVALID
    assert att(n_kv=0) == INVALID
    assert att(q=MISALIGNED) == INVALID
    assert att(table=FAKE, max_pages=0, kv_page=64) == INVALID                 # paged needs max_pages
    assert att(ws=None) == WORKSPACE                                           # 8 rows: split partials
    # MQA and paged caches expand the runs into a list at the head of the workspace
    need = L.lsa_sparse_attn_runs_workspace_size(ctypes.byref(mqa.c()), 8, 64, 0)
    assert need >= 8 * 64 * 4 + 8 * 4
    assert att(prm=mqa, v=FAKE, wsb=need - 1) == WORKSPACE
    assert L.lsa_sparse_attn_runs_workspace_size(ctypes.byref(mla.c()), 131072, 3076, 0) == 0   # fused, no list
    assert L.lsa_sparse_attn_runs_workspace_size(ctypes.byref(mla.c()), 64, 2308, 1) > 64 * 2308 * 4
    assert att(n_rows=0, q=None, runs=None, rc=None, out=None, ws=None, wsb=0) == OK


def test_bad_split_attention_arguments():
    """lsa_hfa_attn validates on the host before touching streams or events."""
    L = lsa.lib()
    mla = lsa.AttnParams(sm_scale=0.07, **lsa.MLA)

    def hfa(prm=mla, n_rows=8, q=FAKE, kv=FAKE, n_kv=4096, idx=FAKE, cnt=FAKE, k_cap=64, q_start=0, k_swa=32,
            out=FAKE, lse=None, ws=FAKE, wsb=1 << 40):
        return L.lsa_hfa_attn(ctypes.byref(prm.c()), n_rows, q, kv, n_kv, idx, cnt, k_cap, q_start, k_swa, out, lse,
                              ws, wsb, None)
    assert hfa(prm=lsa.AttnParams(sm_scale=0.1, **lsa.MQA)) == UNSUPPORTED     # MLA latent cache only
    assert hfa(q_start=4090) == INVALID                                        # window past the cache
    assert hfa(q_start=(1 << 63) - 4) == INVALID                               # no signed overflow
    assert hfa(k_swa=-1) == INVALID
    assert hfa(k_cap=0) == INVALID
    assert hfa(q=MISALIGNED) == INVALID
    assert hfa(idx=None) == INVALID
    assert hfa(ws=None) == WORKSPACE
    assert hfa(wsb=16) == WORKSPACE
    assert hfa(n_rows=0, q=None, idx=None, cnt=None, out=None, ws=None, wsb=0) == OK
    # two partials per row and head (O normalised, in bf16, and (m, l) in fp32), for at most 16384
    # rows per pass
    assert L.lsa_hfa_attn_workspace_size(ctypes.byref(mla.c()), 100) == 100 * 2 * 64 * (512 * 2 + 2 * 4)
    assert L.lsa_hfa_attn_workspace_size(ctypes.byref(mla.c()), 131072) == 16384 * 2 * 64 * (512 * 2 + 2 * 4)


def test_workspace_sizes():
    L = lsa.lib()
    prm = P()
    n = L.lsa_index_workspace_size(ctypes.byref(prm.c()), 131072, 131072)
    # page scores (1024 per row) + page lists (64 per row) + fine scores (64*128 per row)
    assert n == 131072 * 1024 * 4 + 131072 * 64 * 4 + 131072 * 8192 * 4
    mla = lsa.AttnParams(sm_scale=0.07, **lsa.MLA)
    assert L.lsa_sparse_attn_workspace_size(ctypes.byref(mla.c()), 131072, 3076, 0) == 0
    assert L.lsa_sparse_attn_workspace_size(ctypes.byref(mla.c()), 64, 2308, 1) > 64 * 2308 * 4


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(lsa, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(lsa, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        lsa.lib()


def test_zero_sized_calls_accept_null_buffers():
    """Nothing to read or write: empty tensors (NULL data pointers) are accepted, no launch."""
    L = lsa.lib()
    prm = P()
    assert L.lsa_block_means(ctypes.byref(prm.c()), 64, None, None, None, None) == OK       # 64 < sub_block
    assert prefill(prm, n_q=0, q=None, w=None, idx=None, cnt=None, ws=None, wsb=0) == OK
    mla = lsa.AttnParams(sm_scale=0.07, **lsa.MLA)
    assert L.lsa_sparse_attn(ctypes.byref(mla.c()), 0, None, FAKE, None, 10, None, None, 8, None, 0, 0, 1,
                             None, None, None, 0, None) == OK


def test_binding_refuses_host_tensors():
    """The product path never computes on the CPU: host tensors are refused by the binding before
    the library is called (there is no CPU fallback)."""
    mla = lsa.AttnParams(sm_scale=0.07, **lsa.MLA)
    q = torch.zeros((2, 64, 576), dtype=torch.bfloat16)
    kv = torch.zeros((8, 576), dtype=torch.bfloat16)
    idx = torch.zeros((2, 4), dtype=torch.int32)
    cnt = torch.ones((2,), dtype=torch.int32)
    with pytest.raises(ValueError, match="CUDA"):
        lsa.sparse_attn(mla, q, kv, None, idx, cnt)
    with pytest.raises(ValueError, match="CUDA"):
        lsa.sparse_attn_runs(mla, q, kv, torch.zeros((2, 4, 2), dtype=torch.int32), cnt)
    prm = P()
    with pytest.raises(ValueError, match="CUDA"):
        lsa.index_prefill(prm, torch.zeros((2, prm.n_heads, prm.head_dim), dtype=torch.bfloat16),
                          torch.zeros((2, prm.n_heads)), torch.zeros((8, prm.head_dim), dtype=torch.uint8),
                          torch.ones(8), None, 0)


def test_header_is_plain_c(tmp_path):
    """include/lsa.h is a C header: it compiles as C99 (pedantic) and as C++11."""
    import shutil
    import subprocess
    for cc, std, ext in (("gcc", "-std=c99", "c"), ("g++", "-std=c++11", "cpp")):
        if shutil.which(cc) is None:
            pytest.skip(f"{cc} not available")
        src = tmp_path / f"use.{ext}"
        src.write_text('#include "lsa.h"\nint main(void) { return lsa_version() == 0; }\n')
        r = subprocess.run([cc, std, "-Wall", "-Wextra", "-pedantic", "-Werror", "-fsyntax-only",
                            f"-I{os.path.join(ROOT, 'include')}", str(src)], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr
