"""The C-ABI library: it loads, exports every symbol the header declares, and
rejects bad arguments before any HIP call (so these run without a GPU)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2609_32420_amd as P
from paper_2609_32420_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "carnator.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(P.LIB_PATH):
        B.build()
    return P.lib()


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(carnator_\w+)\s*\(", text)))


def test_header_declares_the_python_export_list():
    assert _declared() == sorted(P.EXPORTS)


def test_every_declared_symbol_is_exported(L):
    out = subprocess.run(["nm", "-D", "--defined-only", P.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT (carnator_\w+)", out))
    for name in _declared():
        assert name in exported, name
        assert getattr(L, name) is not None


def test_abi_version_and_status_strings(L):
    assert L.carnator_abi_version() == P.ABI_VERSION
    declared = re.search(r"#define CARNATOR_ABI_VERSION (\d+)", open(HEADER).read())
    assert int(declared.group(1)) == P.ABI_VERSION
    assert L.carnator_status_str(0) == b"ok"
    for code in (-1, -2, -3, -4, -5, -6):
        assert L.carnator_status_str(code) not in (b"", b"unknown status")
    assert L.carnator_status_str(12345) == b"unknown status"


def _shape(B=1, H=2, N=192, d=64, bs=64):
    return P.Shape(B, H, N, d, bs)


def _view(ptr=0x10000, sb=0, sh=0, sn=64):
    return P.View(ptr, sb, sh, sn)


def test_workspace_sizes(L):
    s = _shape(1, 12, 32760, 128, 128)
    nb = 256
    assert L.carnator_build_block_mask_workspace_size(ctypes.byref(s)) == 2 * 12 * nb * 128 * 8
    ws = L.carnator_block_sparse_attn_workspace_size(ctypes.byref(s))
    assert ws >= 12 * nb * nb * 4 + 3 * 12 * nb * 4
    assert L.carnator_signature_sim_workspace_size(1, 4096, 8) >= 4096 * 8
    bad = _shape(d=96)
    assert L.carnator_block_sparse_attn_workspace_size(ctypes.byref(bad)) == 0


def _err(L):
    return L.carnator_last_error().decode()


@pytest.mark.parametrize("field,value,code", [
    ("head_dim", 96, -3), ("block", 32, -3), ("batch", 0, -2), ("seq_len", 0, -2),
    ("heads", -1, -2), ("seq_len", 2049 * 128, -3)])
def test_build_mask_rejects_shapes(L, field, value, code):
    s = _shape(bs=128, d=128)
    setattr(s, field, value)
    q = _view(sn=128)
    r = L.carnator_build_block_mask(ctypes.byref(q), ctypes.byref(q), ctypes.byref(s), 0.0, 0.9,
                                    ctypes.c_void_p(0x20000), ctypes.c_void_p(0x40000), 1 << 30, None)
    assert r == code and _err(L)


def test_build_mask_rejects_pointers_alignment_threshold_workspace(L):
    s = _shape()
    q = _view()
    dst = ctypes.c_void_p(0x20000)
    ws = ctypes.c_void_p(0x40000)
    call = lambda qv, kv, tau, out, w, n: L.carnator_build_block_mask(
        ctypes.byref(qv) if qv is not None else None, ctypes.byref(kv) if kv is not None else None,
        ctypes.byref(s), 0.0, tau, out, w, n, None)
    assert call(None, q, 0.9, dst, ws, 1 << 30) == -1
    assert call(q, q, 0.9, None, ws, 1 << 30) == -1
    assert call(_view(ptr=0x10008), q, 0.9, dst, ws, 1 << 30) == -4
    assert call(_view(sn=60), q, 0.9, dst, ws, 1 << 30) == -4
    assert call(_view(sn=56), q, 0.9, dst, ws, 1 << 30) == -2
    assert call(q, q, 0.0, dst, ws, 1 << 30) == -2
    assert call(q, q, float("nan"), dst, ws, 1 << 30) == -2
    assert call(q, q, 0.9, dst, None, 1 << 30) == -5
    assert call(q, q, 0.9, dst, ws, 16) == -5
    assert call(q, q, 0.9, dst, ctypes.c_void_p(0x40010), 1 << 30) == -4
    assert "workspace" in _err(L)


def test_attention_rejects_bad_arguments(L):
    s = _shape()
    q = _view()
    out = ctypes.c_void_p(0x20000)
    mask = ctypes.c_void_p(0x30000)
    ws = ctypes.c_void_p(0x40000)

    def call(o=out, osn=64, m=mask, w=ws, n=1 << 30, qv=q, scale=0.0):
        return L.carnator_block_sparse_attn(ctypes.byref(qv), ctypes.byref(q), ctypes.byref(q), o, 0, 0, osn,
                                            ctypes.byref(s), m, scale, None, w, n, None)
    assert call(o=None) == -1
    assert call(m=None) == -1
    assert call(o=ctypes.c_void_p(0x20002)) == -4
    assert call(osn=12) == -4
    assert call(osn=32) == -2
    assert call(w=None) == -5
    assert call(n=100) == -5
    assert call(qv=_view(ptr=0)) == -1
    assert call(scale=float("inf")) == -2
    # a row stride above 2^24 elements overflows the kernel's 32-bit tile
    # offsets: rejected before anything is enqueued
    assert call(qv=_view(sn=(1 << 24) + 8)) == -3
    assert call(qv=_view(sn=1 << 24), n=100) == -5  # the largest accepted stride passes this check


def test_attention_lists_rejects_bad_arguments(L):
    s = _shape()
    q = _view()
    out = ctypes.c_void_p(0x20000)
    p = ctypes.c_void_p(0x30000)

    def call(o=out, osn=64, rp=p, ci=p, od=p, qv=q, scale=0.0, shape=s):
        return L.carnator_block_sparse_attn_lists(ctypes.byref(qv), ctypes.byref(q), ctypes.byref(q), o, 0, 0, osn,
                                                  ctypes.byref(shape), rp, ci, od, scale, None, None)
    assert call(o=None) == -1
    assert call(rp=None) == -1 and call(ci=None) == -1 and call(od=None) == -1
    assert call(o=ctypes.c_void_p(0x20002)) == -4
    assert call(osn=12) == -4
    assert call(scale=float("nan")) == -2
    assert call(shape=_shape(d=96)) == -3
    assert call(qv=_view(sn=(1 << 24) + 8)) == -3
    assert "stride_n" in _err(L)


def test_merge_compact_signature_reject(L):
    s = _shape()
    assert L.carnator_merge_target_rows(None, ctypes.byref(s), ctypes.c_void_p(0x100), None, None) == -1
    assert L.carnator_merge_target_rows(ctypes.c_void_p(0x100), ctypes.byref(s), None, None, None) == -1
    assert L.carnator_merge_target_rows(ctypes.c_void_p(0x100), None, ctypes.c_void_p(0x100), None, None) == -1
    p = ctypes.c_void_p(0x1000)
    assert L.carnator_compact_block_mask(p, ctypes.byref(s), p, None, p, p, 1 << 20, None) == -1
    assert L.carnator_compact_block_mask(p, ctypes.byref(s), p, p, p, p, 4, None) == -5
    q = ctypes.c_void_p(0x10000)
    sig = L.carnator_signature_sim
    assert sig(None, 1, q, 8, 16, 16, 2, q, q, None, q, 1 << 20, None) == -1
    assert sig(q, 1, q, 8, 16, 16, 9, q, q, None, q, 1 << 20, None) == -2
    assert sig(q, 1, q, 100, 16, 16, 65, q, q, None, q, 1 << 20, None) == -3
    assert sig(q, 1, q, 8, 16, 8, 2, q, q, None, q, 1 << 20, None) == -2
    assert sig(q, 1, q, 8, 18, 20, 2, q, q, None, q, 1 << 20, None) == -4
    assert sig(q, 1, q, 8, 16, 16, 2, q, q, None, q, 8, None) == -5
    assert L.carnator_signature_sim_workspace_size(2, 4096, 8) == 2 * 4096 * 8
    # the no-allocation call: same checks, and nq * m bounded by its 4 MiB scratch
    na = L.carnator_signature_sim_noalloc
    assert na(None, 1, q, 8, 16, 16, 2, q, q, None, None) == -1
    assert na(q, 1, q, 8, 16, 16, 9, q, q, None, None) == -2
    assert na(q, 1, q, 100, 16, 16, 65, q, q, None, None) == -3
    assert na(q, 1, q, 8, 18, 20, 2, q, q, None, None) == -4
    assert na(q, 1, q, 524289, 16, 16, 2, q, q, None, None) == -5
    assert na(q, 2, q, 262145, 16, 16, 2, q, q, None, None) == -5
    assert "524288" in _err(L)


def test_python_binding_raises_without_gpu_tensors():
    import torch
    x = torch.zeros(1, 1, 64, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        P.block_sparse_attn(x, x, x, torch.ones(1, 1, 1, 1, dtype=torch.uint8), 64)


def test_bit_packed_entry_points_reject(L):
    s = _shape()
    p = ctypes.c_void_p(0x1000)
    odd = ctypes.c_void_p(0x1004)
    # pack / unpack
    assert L.carnator_pack_block_mask(None, ctypes.byref(s), p, None) == -1
    assert L.carnator_pack_block_mask(p, ctypes.byref(s), None, None) == -1
    assert L.carnator_pack_block_mask(p, ctypes.byref(s), odd, None) == -4
    assert L.carnator_pack_block_mask(p, ctypes.byref(_shape(bs=32)), p, None) == -3
    assert L.carnator_unpack_block_mask(None, ctypes.byref(s), p, None) == -1
    assert L.carnator_unpack_block_mask(odd, ctypes.byref(s), p, None) == -4
    assert L.carnator_unpack_block_mask(p, None, p, None) == -1
    # compaction from bits
    c = L.carnator_compact_block_mask_bits
    assert c(None, ctypes.byref(s), None, None, p, p, p, p, 1 << 20, None) == -1
    assert c(p, ctypes.byref(s), None, None, p, None, p, p, 1 << 20, None) == -1
    assert c(odd, ctypes.byref(s), None, None, p, p, p, p, 1 << 20, None) == -4
    assert c(p, ctypes.byref(s), None, None, p, p, p, p, 4, None) == -5
    assert c(p, ctypes.byref(s), None, None, p, p, p, None, 1 << 20, None) == -5
    assert c(p, ctypes.byref(s), None, None, p, p, p, ctypes.c_void_p(0x1010), 1 << 20, None) == -4
    # builder to bits: the same checks as the uint8 builder, plus bits alignment
    q = _view()
    b = lambda out, tau=0.9, n=1 << 30: L.carnator_build_block_mask_bits(
        ctypes.byref(q), ctypes.byref(q), ctypes.byref(s), 0.0, tau, out, ctypes.c_void_p(0x40000), n, None)
    assert b(None) == -1
    assert b(odd) == -4
    assert b(p, tau=0.0) == -2
    assert b(p, n=16) == -5
    assert "workspace" in _err(L)


def test_order_group_heads(L):
    g = L.carnator_order_group_heads
    # heads whose K and V (2 * N * d bf16 values each) fit 256 MiB
    assert g(ctypes.byref(_shape(1, 12, 32760, 128, 128))) == 12  # 16.8 MB a head: all 12
    assert g(ctypes.byref(_shape(1, 40, 75600, 128, 128))) == 6  # 38.7 MB: 6
    assert g(ctypes.byref(_shape(1, 24, 119056, 128, 128))) == 4  # 61.0 MB: 4
    assert g(ctypes.byref(_shape(2, 24, 119056, 128, 128))) == 4  # groups span the batch
    assert g(ctypes.byref(_shape(1, 200, 262144, 128, 128))) == 4  # 134 MB: 1, but at most 63 groups
    assert g(ctypes.byref(_shape(d=96))) == 0
    assert g(None) == 0


def test_bit_packed_workspace_size(L):
    s = _shape(1, 12, 32760, 128, 128)
    R = 12 * 256
    # the list lengths, the sort's chunk histograms ((nB + 2) keys x at most
    # 3 + 63 chunks of 1024 rows: the rows of up to 63 head groups), chunk
    # offsets, in-chunk prefixes of the lengths and per-group key totals (63
    # groups x (nB + 1) keys), then the packed dense-column words of each
    # batch entry
    a = lambda n: -(-n // 256) * 256
    chunks = 3 + 63
    want = a(R * 4) + a(258 * chunks * 4) + a(chunks * 4) + a(R * 4) + a(63 * 257 * 4) + a(8)
    assert L.carnator_compact_block_mask_bits_workspace_size(ctypes.byref(s)) == want
    assert L.carnator_compact_block_mask_bits_workspace_size(ctypes.byref(_shape(d=96))) == 0
    assert R * 4 == 12288


def test_region_entry_points_reject(L):
    p = ctypes.c_void_p(0x1000)
    ws = ctypes.c_void_p(0x40000)
    rw = L.carnator_region_weights
    assert rw(None, 1, 2, 8, 8, 2, 3, p, p, ws, 1 << 20, None) == -1
    assert rw(p, 0, 2, 8, 8, 2, 3, p, p, ws, 1 << 20, None) == -2
    assert rw(p, 1, 2, 8, 8, -1, 3, p, p, ws, 1 << 20, None) == -2
    assert rw(p, 1, 2, 8, 8, 200, 51, p, p, ws, 1 << 20, None) == -2
    assert rw(p, 1, 2, 300, 300, 2, 3, p, p, ws, 1 << 30, None) == -3
    assert rw(p, 1, 2, 8, 8, 2, 3, p, p, ws, 16, None) == -5
    assert rw(p, 1, 2, 8, 8, 2, 3, p, ctypes.c_void_p(0x1002), ws, 1 << 20, None) == -4
    assert L.carnator_region_weights_workspace_size(1, 2, 8, 8) >= 2 * 64 + 2 * 4
    assert L.carnator_region_weights_workspace_size(0, 2, 8, 8) == 0
    lf = L.carnator_latent_fusion
    assert lf(p, p, p, None, 1, 16, 4, 8, 8, 1, 2, 2, None) == -1
    assert lf(p, p, p, p, 1, 16, 4, 8, 8, 1, 3, 2, None) == -2
    assert lf(p, p, p, p, 1, 16, 4, 8, 8, 0, 2, 2, None) == -2
    assert lf(p, ctypes.c_void_p(0x1001), p, p, 1, 16, 4, 8, 8, 1, 2, 2, None) == -4
    s = _shape(1, 1, 200, 64, 64)
    bf = L.carnator_region_block_flags
    assert bf(None, 0, ctypes.byref(s), p, p, None) == -1
    assert bf(p, 200, ctypes.byref(s), p, p, None) == -2
    assert bf(p, -1, ctypes.byref(s), p, p, None) == -2
    cr = L.carnator_compact_block_mask_bits_region
    assert cr(p, ctypes.byref(s), p, p, p, p, p, None, ws, 1 << 20, None) == -1
    assert cr(p, ctypes.byref(s), None, p, p, p, p, p, ws, 1 << 20, None) == -1
    assert cr(p, ctypes.byref(s), p, p, p, p, p, p, ws, 4, None) == -5
    q = _view()
    ar = L.carnator_block_sparse_attn_rows
    assert ar(ctypes.byref(q), ctypes.byref(q), ctypes.byref(q), ctypes.c_void_p(0x20000), 0, 0, 64,
              ctypes.byref(_shape()), p, p, p, None, 0.0, None, None) == -1


def test_exact_mass_entry_points_reject(L):
    s = _shape()
    q = _view()
    p = ctypes.c_void_p(0x20000)
    ws = ctypes.c_void_p(0x40000)
    m = L.carnator_block_mass_exact
    assert m(ctypes.byref(q), ctypes.byref(q), ctypes.byref(s), 0.0, None, ws, 1 << 30, None) == -1
    assert m(ctypes.byref(q), ctypes.byref(q), ctypes.byref(s), 0.0, ctypes.c_void_p(0x20004), ws, 1 << 30,
             None) == -4
    assert m(ctypes.byref(q), ctypes.byref(q), ctypes.byref(s), 0.0, p, ws, 16, None) == -5
    assert m(ctypes.byref(q), ctypes.byref(q), ctypes.byref(s), float("inf"), p, ws, 1 << 30, None) == -2
    # one 8-byte record per (query, key block) and a 4-byte log-sum-exp per query
    big = _shape(1, 12, 32760, 128, 128)
    assert L.carnator_block_mass_exact_workspace_size(ctypes.byref(big)) >= 12 * 32760 * (256 * 8 + 4)
    # heads in chunks whose records fit in 4 GiB: 4 of 24 heads at 119,056
    # tokens (21 GB for all of them), one head beyond the cap at the largest N
    cap = 4 << 30
    per = 119056 * (931 * 8 + 4)
    hv = _shape(1, 24, 119056, 128, 128)
    need = L.carnator_block_mass_exact_workspace_size(ctypes.byref(hv))
    assert 4 * per <= need <= cap and need < 5 * per
    one = _shape(1, 3, 2048 * 128, 128, 128)
    need1 = L.carnator_block_mass_exact_workspace_size(ctypes.byref(one))
    assert 2048 * 128 * (2048 * 8 + 4) <= need1 < 2 * 2048 * 128 * (2048 * 8 + 4)
    # a workspace one byte short of the chunked size is rejected before any launch
    qv = _view(sn=128)
    assert m(ctypes.byref(qv), ctypes.byref(qv), ctypes.byref(hv), 0.0, p, ws, need - 1, None) == -5
    assert "workspace" in _err(L)
    sel = L.carnator_select_block_mask
    assert sel(None, ctypes.byref(s), 0.9, p, None, None) == -1
    assert sel(p, ctypes.byref(s), 0.9, None, None, None) == -1
    assert sel(p, ctypes.byref(s), 0.9, p, p, None) == -1
    assert sel(p, ctypes.byref(s), 0.0, p, None, None) == -2
    assert sel(ctypes.c_void_p(0x20004), ctypes.byref(s), 0.9, p, None, None) == -4
