"""Python binding of libcarnator (the C ABI in include/carnator.h).

Argument marshalling only: every step of the path runs in the HIP kernels of
libcarnator.so.  Tensors live on the GPU (PyTorch provides device memory and
the current stream); outputs and workspaces are allocated with torch.empty.
There is no CPU fallback: if the library is missing, importing the functions
works but every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libcarnator.so")

CARNATOR_OK = 0
# CARNATOR_ABI_VERSION of include/carnator.h this binding marshals for
ABI_VERSION = 7
STATUS = {0: "OK", -1: "E_NULL", -2: "E_SHAPE", -3: "E_UNSUPPORTED", -4: "E_ALIGN",
          -5: "E_WORKSPACE", -6: "E_HIP"}

# Every entry point declared in include/carnator.h.
EXPORTS = (
    "carnator_abi_version", "carnator_status_str", "carnator_last_error", "carnator_order_group_heads",
    "carnator_build_block_mask_workspace_size", "carnator_build_block_mask",
    "carnator_merge_target_rows",
    "carnator_block_mass_exact_workspace_size", "carnator_block_mass_exact", "carnator_select_block_mask",
    "carnator_compact_block_mask_workspace_size", "carnator_compact_block_mask",
    "carnator_build_block_mask_bits", "carnator_pack_block_mask", "carnator_unpack_block_mask",
    "carnator_compact_block_mask_bits_workspace_size", "carnator_compact_block_mask_bits",
    "carnator_region_weights_workspace_size", "carnator_region_weights", "carnator_latent_fusion",
    "carnator_region_block_flags", "carnator_compact_block_mask_bits_region",
    "carnator_block_sparse_attn_rows",
    "carnator_block_sparse_attn_workspace_size", "carnator_block_sparse_attn",
    "carnator_block_sparse_attn_lists",
    "carnator_signature_sim_workspace_size", "carnator_signature_sim", "carnator_signature_sim_noalloc",
    "carnator_ciede2000", "carnator_shape_descriptor", "carnator_object_discrepancy", "carnator_compat_gate",
    "carnator_clopper_pearson_upper",
)


class Shape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("heads", ctypes.c_int32), ("seq_len", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("block", ctypes.c_int32)]


class View(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("stride_b", ctypes.c_int64), ("stride_h", ctypes.c_int64),
                ("stride_n", ctypes.c_int64)]


class CarnatorError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__("%s (%d): %s" % (STATUS.get(status, "?"), status, detail))
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libcarnator.so is not built (run python -m paper_2609_32420_amd.build)")
        L = ctypes.CDLL(LIB_PATH)
        P, I32, I64, SZ, F32, F64 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t,
                                     ctypes.c_float, ctypes.c_double)
        SP, VP = ctypes.POINTER(Shape), ctypes.POINTER(View)
        sig = {
            "carnator_abi_version": (ctypes.c_int, []),
            "carnator_order_group_heads": (ctypes.c_int32, [ctypes.POINTER(Shape)]),
            "carnator_status_str": (ctypes.c_char_p, [ctypes.c_int]),
            "carnator_last_error": (ctypes.c_char_p, []),
            "carnator_build_block_mask_workspace_size": (SZ, [SP]),
            "carnator_build_block_mask": (ctypes.c_int, [VP, VP, SP, F32, F64, P, P, SZ, P]),
            "carnator_merge_target_rows": (ctypes.c_int, [P, SP, P, P, P]),
            "carnator_block_mass_exact_workspace_size": (SZ, [SP]),
            "carnator_block_mass_exact": (ctypes.c_int, [VP, VP, SP, F32, P, P, SZ, P]),
            "carnator_select_block_mask": (ctypes.c_int, [P, SP, F64, P, P, P]),
            "carnator_compact_block_mask_workspace_size": (SZ, [SP]),
            "carnator_compact_block_mask": (ctypes.c_int, [P, SP, P, P, P, P, SZ, P]),
            "carnator_build_block_mask_bits": (ctypes.c_int, [VP, VP, SP, F32, F64, P, P, SZ, P]),
            "carnator_pack_block_mask": (ctypes.c_int, [P, SP, P, P]),
            "carnator_unpack_block_mask": (ctypes.c_int, [P, SP, P, P]),
            "carnator_compact_block_mask_bits_workspace_size": (SZ, [SP]),
            "carnator_compact_block_mask_bits": (ctypes.c_int, [P, SP, P, P, P, P, P, P, SZ, P]),
            "carnator_region_weights_workspace_size": (SZ, [I32, I32, I32, I32]),
            "carnator_region_weights": (ctypes.c_int, [P, I32, I32, I32, I32, I32, I32, P, P, P, SZ, P]),
            "carnator_latent_fusion": (ctypes.c_int, [P, P, P, P, I32, I32, I32, I32, I32, I32, I32, I32, P]),
            "carnator_region_block_flags": (ctypes.c_int, [P, I32, SP, P, P, P]),
            "carnator_compact_block_mask_bits_region": (ctypes.c_int, [P, SP, P, P, P, P, P, P, P, SZ, P]),
            "carnator_block_sparse_attn_rows": (ctypes.c_int, [VP, VP, VP, P, I64, I64, I64, SP, P, P, P, P,
                                                               F32, P, P]),
            "carnator_block_sparse_attn_workspace_size": (SZ, [SP]),
            "carnator_block_sparse_attn": (ctypes.c_int, [VP, VP, VP, P, I64, I64, I64, SP, P, F32, P, P,
                                                          SZ, P]),
            "carnator_block_sparse_attn_lists": (ctypes.c_int, [VP, VP, VP, P, I64, I64, I64, SP, P, P, P, F32,
                                                                P, P]),
            "carnator_signature_sim_workspace_size": (SZ, [I64, I64, I32]),
            "carnator_signature_sim": (ctypes.c_int, [P, I64, P, I64, I64, I64, I32, P, P, P, P, SZ, P]),
            "carnator_signature_sim_noalloc": (ctypes.c_int, [P, I64, P, I64, I64, I64, I32, P, P, P, P]),
            "carnator_ciede2000": (ctypes.c_int, [P, P, I64, P]),
            "carnator_shape_descriptor": (ctypes.c_int, [P, I32, I32, I32, P, P]),
            "carnator_object_discrepancy": (ctypes.c_int, [F64, F64, P, P, I32, P, P, P]),
            "carnator_compat_gate": (ctypes.c_int, [P, I64, I32, P, P]),
            "carnator_clopper_pearson_upper": (ctypes.c_int, [I64, I64, F64, P]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        if L.carnator_abi_version() != ABI_VERSION:
            raise RuntimeError("libcarnator.so has ABI version %d, the binding expects %d (rebuild it)"
                               % (L.carnator_abi_version(), ABI_VERSION))
        _lib = L
    return _lib


def _check(status: int):
    if status != CARNATOR_OK:
        raise CarnatorError(status, lib().carnator_last_error().decode())


def _stream(t: torch.Tensor):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _shape(t: torch.Tensor, block: int) -> Shape:
    B, H, N, d = t.shape
    return Shape(B, H, N, d, block)


def _mask_shape(B: int, H: int, nb: int, attn=None) -> Shape:
    """Shape of a call on block masks alone.  ``attn`` = (seq_len, head_dim,
    block) of the attention the lists serve sets the head groups of the row
    order (order_group_heads); without it the shape is seq_len nb * 64,
    head_dim 64, block 64."""
    if attn is None:
        return Shape(B, H, nb * 64, 64, 64)
    N, d, bs = (int(x) for x in attn)
    if -(-N // bs) != nb:
        raise ValueError("attn (seq_len %d, block %d) gives %d blocks, the mask has %d" % (N, bs, -(-N // bs), nb))
    return Shape(B, H, N, d, bs)


def order_group_heads(batch: int, heads: int, nb: int, attn=None) -> int:
    """Heads per group of the row order the compaction calls write for masks
    [batch, heads, nb, nb] (carnator_order_group_heads; ``attn`` as in the
    compaction calls)."""
    s = _mask_shape(batch, heads, nb, attn)
    g = lib().carnator_order_group_heads(ctypes.byref(s))
    if g <= 0:
        raise ValueError("invalid shape")
    return int(g)


def _view(t: torch.Tensor) -> View:
    if t.dim() != 4 or t.dtype != torch.bfloat16 or not t.is_cuda or t.stride(3) != 1:
        raise ValueError("expected a bf16 CUDA tensor [B, H, N, d] with d contiguous")
    return View(t.data_ptr(), t.stride(0), t.stride(1), t.stride(2))


def _workspace(nbytes: int, device) -> torch.Tensor:
    # torch's caching allocator returns blocks aligned to at least 512 bytes
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def _dev_u8(x, device, shape) -> Optional[torch.Tensor]:
    if x is None:
        return None
    x = torch.as_tensor(x, device=device)
    if x.dtype != torch.uint8:
        x = (x != 0).to(torch.uint8)
    x = x.contiguous()
    if tuple(x.shape) != tuple(shape):
        raise ValueError("flags must have shape %s" % (tuple(shape),))
    return x


def abi_version() -> int:
    return lib().carnator_abi_version()


def build_block_mask_workspace(q_hist: torch.Tensor, block: int) -> torch.Tensor:
    s = _shape(q_hist, block)
    return _workspace(lib().carnator_build_block_mask_workspace_size(ctypes.byref(s)), q_hist.device)


def build_block_mask(q_hist: torch.Tensor, k_hist: torch.Tensor, block: int, mass_threshold: float,
                     scale: float = 0.0, out: Optional[torch.Tensor] = None,
                     workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Historical block mask uint8 [B, H, nB, nB] (carnator_build_block_mask)."""
    s = _shape(q_hist, block)
    if tuple(k_hist.shape) != tuple(q_hist.shape):
        raise ValueError("q_hist and k_hist shapes differ")
    nb = -(-s.seq_len // block)
    if out is None:
        out = torch.empty(s.batch, s.heads, nb, nb, dtype=torch.uint8, device=q_hist.device)
    L = lib()
    ws = workspace if workspace is not None else build_block_mask_workspace(q_hist, block)
    qv, kv = _view(q_hist), _view(k_hist)
    _check(L.carnator_build_block_mask(ctypes.byref(qv), ctypes.byref(kv), ctypes.byref(s), float(scale),
                                       float(mass_threshold), _ptr(out), _ptr(ws), ws.numel(),
                                       _stream(q_hist)))
    return out


def block_mass_exact(q_hist: torch.Tensor, k_hist: torch.Tensor, block: int, scale: float = 0.0,
                     out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Token-level attention mass of every block pair, fp64 [B, H, nB, nB]
    (carnator_block_mass_exact)."""
    s = _shape(q_hist, block)
    if tuple(k_hist.shape) != tuple(q_hist.shape):
        raise ValueError("q_hist and k_hist shapes differ")
    nb = -(-s.seq_len // block)
    if out is None:
        out = torch.empty(s.batch, s.heads, nb, nb, dtype=torch.float64, device=q_hist.device)
    if out.dtype != torch.float64 or not out.is_contiguous() or tuple(out.shape) != (s.batch, s.heads, nb, nb):
        raise ValueError("out must be a contiguous fp64 [B, H, nB, nB] tensor")
    L = lib()
    if workspace is None:
        workspace = _workspace(L.carnator_block_mass_exact_workspace_size(ctypes.byref(s)), q_hist.device)
    qv, kv = _view(q_hist), _view(k_hist)
    _check(L.carnator_block_mass_exact(ctypes.byref(qv), ctypes.byref(kv), ctypes.byref(s), float(scale), _ptr(out),
                                       _ptr(workspace), workspace.numel(), _stream(q_hist)))
    return out


def select_block_mask(mass: torch.Tensor, mass_threshold: float, bits: bool = False,
                      out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Top-mass selection on given masses fp64 [B, H, nB, nB]: uint8 mask, or
    the packed int64 [B, H, nB, W] with bits=True (carnator_select_block_mask)."""
    if mass.dim() != 4 or mass.dtype != torch.float64 or not mass.is_contiguous():
        raise ValueError("mass must be a contiguous fp64 [B, H, nB, nB] tensor")
    B, H, nb, _ = mass.shape
    if out is None:
        out = (torch.empty(B, H, nb, mask_words(nb), dtype=torch.int64, device=mass.device) if bits
               else torch.empty(B, H, nb, nb, dtype=torch.uint8, device=mass.device))
    s = Shape(B, H, nb * 64, 64, 64)
    _check(lib().carnator_select_block_mask(_ptr(mass), ctypes.byref(s), float(mass_threshold),
                                            None if bits else _ptr(out), _ptr(out) if bits else None,
                                            _stream(mass)))
    return out


def merge_target_rows(mask: torch.Tensor, target_rows, dense_cols=None) -> torch.Tensor:
    """Widens flagged query blocks to full rows (and flagged key blocks to full
    columns) in place; returns ``mask``."""
    B, H, nb, nb2 = mask.shape
    if mask.dtype != torch.uint8 or not mask.is_contiguous() or nb != nb2:
        raise ValueError("mask must be a contiguous uint8 [B, H, nB, nB] tensor")
    rows = _dev_u8(target_rows, mask.device, (B, nb))
    cols = _dev_u8(dense_cols, mask.device, (B, nb))
    # any seq_len with this block count and a supported block size describes the mask
    s = Shape(B, H, nb * 64, 64, 64)
    _check(lib().carnator_merge_target_rows(_ptr(mask), ctypes.byref(s), _ptr(rows), _ptr(cols),
                                            _stream(mask)))
    return mask


def compact_block_mask_workspace(mask: torch.Tensor) -> torch.Tensor:
    B, H, nb, _ = mask.shape
    s = Shape(B, H, nb * 64, 64, 64)
    return _workspace(lib().carnator_compact_block_mask_workspace_size(ctypes.byref(s)), mask.device)


def compact_block_mask(mask: torch.Tensor, trim: bool = True, out=None,
                       workspace: Optional[torch.Tensor] = None, attn=None):
    """(row_ptr int32 [R+1], col_idx int32, order int32 [R]).

    With trim (the default) the stream is synchronised once to cut col_idx to
    its nnz entries; trim=False keeps the full B*H*nB*nB capacity and does not
    synchronise.  ``out`` may pass preallocated (row_ptr, col_idx, order).
    ``attn`` = (seq_len, head_dim, block) of the attention the lists serve: it
    sets the head groups of the order (see order_group_heads).
    """
    B, H, nb, _ = mask.shape
    R = B * H * nb
    s = _mask_shape(B, H, nb, attn)
    dev = mask.device
    if not mask.is_contiguous() or mask.dtype != torch.uint8:
        raise ValueError("mask must be contiguous uint8 [B, H, nB, nB]")
    if out is None:
        out = (torch.empty(R + 1, dtype=torch.int32, device=dev),
               torch.empty(max(R * nb, 1), dtype=torch.int32, device=dev),
               torch.empty(R, dtype=torch.int32, device=dev))
    row_ptr, col_idx, order = out
    if row_ptr.numel() < R + 1 or col_idx.numel() < R * nb or order.numel() < R:
        raise ValueError("out tensors too small")
    L = lib()
    if workspace is None:
        workspace = compact_block_mask_workspace(mask)
    _check(L.carnator_compact_block_mask(_ptr(mask), ctypes.byref(s), _ptr(row_ptr), _ptr(col_idx), _ptr(order),
                                         _ptr(workspace), workspace.numel(), _stream(mask)))
    if trim:
        nnz = int(row_ptr[-1].item())
        return row_ptr, col_idx[:nnz], order
    return row_ptr, col_idx, order


# ---------------------------------------------------------------- bit-packed masks
#
# A packed mask is an int64 tensor [B, H, nB, W], W = ceil(nB / 64), holding
# the uint64 words of include/carnator.h (torch has no general uint64 device
# arithmetic; the bits are the same).


def mask_words(nb: int) -> int:
    """Words per packed mask row."""
    return (nb + 63) // 64


def _bits_shape(bits: torch.Tensor):
    if bits.dim() != 4 or bits.dtype != torch.int64 or not bits.is_contiguous():
        raise ValueError("bits must be a contiguous int64 [B, H, nB, W] tensor")
    B, H, nb, w = bits.shape
    if w != mask_words(nb):
        raise ValueError("bits has %d words per row; nB = %d needs %d" % (w, nb, mask_words(nb)))
    return B, H, nb


def build_block_mask_bits(q_hist: torch.Tensor, k_hist: torch.Tensor, block: int, mass_threshold: float,
                          scale: float = 0.0, out: Optional[torch.Tensor] = None,
                          workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Historical block mask, bit-packed: int64 [B, H, nB, W]
    (carnator_build_block_mask_bits)."""
    s = _shape(q_hist, block)
    if tuple(k_hist.shape) != tuple(q_hist.shape):
        raise ValueError("q_hist and k_hist shapes differ")
    nb = -(-s.seq_len // block)
    if out is None:
        out = torch.empty(s.batch, s.heads, nb, mask_words(nb), dtype=torch.int64, device=q_hist.device)
    elif tuple(out.shape) != (s.batch, s.heads, nb, mask_words(nb)):
        raise ValueError("out must have shape %s" % ((s.batch, s.heads, nb, mask_words(nb)),))
    _bits_shape(out)
    L = lib()
    ws = workspace if workspace is not None else build_block_mask_workspace(q_hist, block)
    qv, kv = _view(q_hist), _view(k_hist)
    _check(L.carnator_build_block_mask_bits(ctypes.byref(qv), ctypes.byref(kv), ctypes.byref(s), float(scale),
                                            float(mass_threshold), _ptr(out), _ptr(ws), ws.numel(),
                                            _stream(q_hist)))
    return out


def pack_block_mask(mask: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """uint8 [B, H, nB, nB] -> packed int64 [B, H, nB, W]."""
    B, H, nb, nb2 = mask.shape
    if mask.dtype != torch.uint8 or not mask.is_contiguous() or nb != nb2:
        raise ValueError("mask must be a contiguous uint8 [B, H, nB, nB] tensor")
    if out is None:
        out = torch.empty(B, H, nb, mask_words(nb), dtype=torch.int64, device=mask.device)
    if _bits_shape(out) != (B, H, nb):
        raise ValueError("out must have shape %s" % ((B, H, nb, mask_words(nb)),))
    s = Shape(B, H, nb * 64, 64, 64)
    _check(lib().carnator_pack_block_mask(_ptr(mask), ctypes.byref(s), _ptr(out), _stream(mask)))
    return out


def unpack_block_mask(bits: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Packed int64 [B, H, nB, W] -> uint8 [B, H, nB, nB] of 0/1."""
    B, H, nb = _bits_shape(bits)
    if out is None:
        out = torch.empty(B, H, nb, nb, dtype=torch.uint8, device=bits.device)
    if out.dtype != torch.uint8 or not out.is_contiguous() or tuple(out.shape) != (B, H, nb, nb):
        raise ValueError("out must be a contiguous uint8 %s tensor" % ((B, H, nb, nb),))
    s = Shape(B, H, nb * 64, 64, 64)
    _check(lib().carnator_unpack_block_mask(_ptr(bits), ctypes.byref(s), _ptr(out), _stream(bits)))
    return out


def compact_block_mask_bits_workspace(bits: torch.Tensor) -> torch.Tensor:
    B, H, nb = _bits_shape(bits)
    s = Shape(B, H, nb * 64, 64, 64)
    return _workspace(lib().carnator_compact_block_mask_bits_workspace_size(ctypes.byref(s)), bits.device)


def compact_block_mask_bits(bits: torch.Tensor, target_rows=None, dense_cols=None, trim: bool = True,
                            out=None, workspace: Optional[torch.Tensor] = None, attn=None):
    """(row_ptr, col_idx, order) of the packed mask widened by target_rows and
    dense_cols (each [B, nB] or None); the bits are not modified.  trim, out
    and attn as in compact_block_mask."""
    B, H, nb = _bits_shape(bits)
    R = B * H * nb
    dev = bits.device
    rows = _dev_u8(target_rows, dev, (B, nb))
    cols = _dev_u8(dense_cols, dev, (B, nb))
    s = _mask_shape(B, H, nb, attn)
    if out is None:
        out = (torch.empty(R + 1, dtype=torch.int32, device=dev),
               torch.empty(max(R * nb, 1), dtype=torch.int32, device=dev),
               torch.empty(R, dtype=torch.int32, device=dev))
    row_ptr, col_idx, order = out
    if row_ptr.numel() < R + 1 or col_idx.numel() < R * nb or order.numel() < R:
        raise ValueError("out tensors too small")
    if workspace is None:
        workspace = compact_block_mask_bits_workspace(bits)
    _check(lib().carnator_compact_block_mask_bits(_ptr(bits), ctypes.byref(s), _ptr(rows), _ptr(cols),
                                                  _ptr(row_ptr), _ptr(col_idx), _ptr(order), _ptr(workspace),
                                                  workspace.numel(), _stream(bits)))
    if trim:
        nnz = int(row_ptr[-1].item())
        return row_ptr, col_idx[:nnz], order
    return row_ptr, col_idx, order


class MaskBank:
    """The reused connectivity of one historical request: a packed block mask
    per (denoising step, guidance branch, layer), each [B, H, nB, W], in one
    int64 array [steps, branches, layers, B, H, nB, W] on the device."""

    def __init__(self, steps: int, branches: int, layers: int, batch: int, heads: int, n_blocks: int,
                 device="cuda"):
        self.n_blocks = n_blocks
        self.bits = torch.zeros(steps, branches, layers, batch, heads, n_blocks, mask_words(n_blocks),
                                dtype=torch.int64, device=device)

    @property
    def nbytes(self) -> int:
        return self.bits.numel() * 8

    def slot(self, step: int, branch: int, layer: int) -> torch.Tensor:
        return self.bits[step, branch, layer]

    def record(self, step: int, branch: int, layer: int, q_hist: torch.Tensor, k_hist: torch.Tensor,
               block: int, mass_threshold: float, scale: float = 0.0,
               workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
        """Builds the historical mask of one slot straight into the bank."""
        return build_block_mask_bits(q_hist, k_hist, block, mass_threshold, scale,
                                     out=self.slot(step, branch, layer), workspace=workspace)

    def store(self, step: int, branch: int, layer: int, mask: torch.Tensor) -> torch.Tensor:
        """Packs a uint8 mask into one slot."""
        return pack_block_mask(mask, out=self.slot(step, branch, layer))

    def lists(self, step: int, branch: int, layer: int, target_rows=None, dense_cols=None,
              trim: bool = True, out=None, workspace: Optional[torch.Tensor] = None, attn=None):
        """Compacted lists of one slot for a target (compact_block_mask_bits;
        attn as there)."""
        return compact_block_mask_bits(self.slot(step, branch, layer), target_rows, dense_cols, trim=trim,
                                       out=out, workspace=workspace, attn=attn)


def block_sparse_attn_workspace(q: torch.Tensor, block: int) -> torch.Tensor:
    s = _shape(q, block)
    return _workspace(lib().carnator_block_sparse_attn_workspace_size(ctypes.byref(s)), q.device)


def block_sparse_attn(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, mask: torch.Tensor, block: int,
                      scale: float = 0.0, return_lse: bool = False, out: Optional[torch.Tensor] = None,
                      workspace: Optional[torch.Tensor] = None):
    """O = softmax(scale q k^T) v restricted to the kept block pairs
    (carnator_block_sparse_attn).  Returns O (and the fp32 LSE)."""
    s = _shape(q, block)
    for t, n in ((k, "k"), (v, "v")):
        if tuple(t.shape) != tuple(q.shape):
            raise ValueError("%s shape differs from q" % n)
    nb = -(-s.seq_len // block)
    if tuple(mask.shape) != (s.batch, s.heads, nb, nb) or mask.dtype != torch.uint8 or not mask.is_contiguous():
        raise ValueError("mask must be contiguous uint8 [B, H, nB, nB]")
    if out is None:
        out = torch.empty_like(q, memory_format=torch.contiguous_format)
    lse = torch.empty(s.batch, s.heads, s.seq_len, dtype=torch.float32, device=q.device) if return_lse else None
    L = lib()
    if workspace is None:
        workspace = block_sparse_attn_workspace(q, block)
    qv, kv, vv = _view(q), _view(k), _view(v)
    _check(L.carnator_block_sparse_attn(ctypes.byref(qv), ctypes.byref(kv), ctypes.byref(vv), _ptr(out),
                                        out.stride(0), out.stride(1), out.stride(2), ctypes.byref(s),
                                        _ptr(mask), float(scale), _ptr(lse), _ptr(workspace),
                                        workspace.numel(), _stream(q)))
    return (out, lse) if return_lse else out


def block_sparse_attn_lists(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, lists, block: int,
                            scale: float = 0.0, return_lse: bool = False, out: Optional[torch.Tensor] = None,
                            n_rows: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None):
    """block_sparse_attn with the mask given as the (row_ptr, col_idx, order)
    lists of compact_block_mask (carnator_block_sparse_attn_lists).  With
    ``n_rows`` (a device int32 tensor of one element) only the rows
    order[0 .. n_rows) are computed (carnator_block_sparse_attn_rows); the
    rest of ``out`` (and of ``lse``, which may be passed in) is untouched."""
    s = _shape(q, block)
    for t, n in ((k, "k"), (v, "v")):
        if tuple(t.shape) != tuple(q.shape):
            raise ValueError("%s shape differs from q" % n)
    row_ptr, col_idx, order = lists
    nb = -(-s.seq_len // block)
    R = s.batch * s.heads * nb
    for t, n, need in ((row_ptr, "row_ptr", R + 1), (order, "order", R)):
        if t.dtype != torch.int32 or not t.is_cuda or t.numel() < need:
            raise ValueError("%s must be int32 on the GPU with at least %d entries" % (n, need))
    if col_idx.dtype != torch.int32 or not col_idx.is_cuda:
        raise ValueError("col_idx must be int32 on the GPU")
    if out is None:
        out = torch.empty_like(q, memory_format=torch.contiguous_format)
    if return_lse and lse is None:
        lse = torch.empty(s.batch, s.heads, s.seq_len, dtype=torch.float32, device=q.device)
    if not return_lse:
        lse = None
    elif lse.dtype != torch.float32 or not lse.is_contiguous() or tuple(lse.shape) != (s.batch, s.heads, s.seq_len):
        raise ValueError("lse must be a contiguous fp32 [B, H, N] tensor")
    qv, kv, vv = _view(q), _view(k), _view(v)
    if n_rows is None:
        _check(lib().carnator_block_sparse_attn_lists(ctypes.byref(qv), ctypes.byref(kv), ctypes.byref(vv),
                                                      _ptr(out), out.stride(0), out.stride(1), out.stride(2),
                                                      ctypes.byref(s), _ptr(row_ptr), _ptr(col_idx), _ptr(order),
                                                      float(scale), _ptr(lse), _stream(q)))
    else:
        if n_rows.dtype != torch.int32 or not n_rows.is_cuda or n_rows.numel() < 1:
            raise ValueError("n_rows must be an int32 GPU tensor")
        _check(lib().carnator_block_sparse_attn_rows(ctypes.byref(qv), ctypes.byref(kv), ctypes.byref(vv),
                                                     _ptr(out), out.stride(0), out.stride(1), out.stride(2),
                                                     ctypes.byref(s), _ptr(row_ptr), _ptr(col_idx), _ptr(order),
                                                     _ptr(n_rows), float(scale), _ptr(lse), _stream(q)))
    return (out, lse) if return_lse else out


# ---------------------------------------------------------------- region-restricted reuse

def region_weights(evidence: torch.Tensor, r_active: int = 2, r_context: int = 3, out=None,
                   workspace: Optional[torch.Tensor] = None):
    """(region codes uint8, W fp32), both [B, T, H, W], from the evidence
    uint8 [B, T, H, W] (carnator_region_weights)."""
    if evidence.dim() != 4 or evidence.dtype != torch.uint8 or not evidence.is_contiguous():
        raise ValueError("evidence must be a contiguous uint8 [B, T, H, W] tensor")
    B, T, H, W = evidence.shape
    dev = evidence.device
    if out is None:
        out = (torch.empty(B, T, H, W, dtype=torch.uint8, device=dev),
               torch.empty(B, T, H, W, dtype=torch.float32, device=dev))
    region, weight = out
    if workspace is None:
        workspace = _workspace(lib().carnator_region_weights_workspace_size(B, T, H, W), dev)
    _check(lib().carnator_region_weights(_ptr(evidence), B, T, H, W, int(r_active), int(r_context), _ptr(region),
                                         _ptr(weight), _ptr(workspace), workspace.numel(), _stream(evidence)))
    return region, weight


def latent_fusion(z_target: torch.Tensor, z_hist: torch.Tensor, weight: torch.Tensor, out=None):
    """W * z_target + (1 - W) * z_hist for fp32 latents [B, C, T, H, W] and W
    on the token grid [B, T/pt, H/ph, W/pw] (carnator_latent_fusion).  ``out``
    may be z_target or z_hist."""
    for t, n in ((z_target, "z_target"), (z_hist, "z_hist")):
        if t.dim() != 5 or t.dtype != torch.float32 or not t.is_contiguous():
            raise ValueError("%s must be a contiguous fp32 [B, C, T, H, W] tensor" % n)
    if tuple(z_hist.shape) != tuple(z_target.shape):
        raise ValueError("z_hist shape differs from z_target")
    if weight.dim() != 4 or weight.dtype != torch.float32 or not weight.is_contiguous():
        raise ValueError("weight must be a contiguous fp32 [B, T, H, W] tensor")
    B, C, T, H, W = z_target.shape
    if weight.shape[0] != B or T % weight.shape[1] or H % weight.shape[2] or W % weight.shape[3]:
        raise ValueError("the weight grid must divide the latent grid")
    pt, ph, pw = T // weight.shape[1], H // weight.shape[2], W // weight.shape[3]
    if out is None:
        out = torch.empty_like(z_target)
    _check(lib().carnator_latent_fusion(_ptr(z_target), _ptr(z_hist), _ptr(weight), _ptr(out), B, C, T, H, W,
                                        pt, ph, pw, _stream(z_target)))
    return out


def region_block_flags(region: torch.Tensor, n_text: int, block: int, out=None):
    """(active query blocks, context key blocks), uint8 [B, nB] each, from the
    region codes [B, T, H, W] of the video tokens (carnator_region_block_flags)."""
    if region.dtype != torch.uint8 or not region.is_contiguous():
        raise ValueError("region must be a contiguous uint8 tensor")
    B = region.shape[0]
    N = n_text + region[0].numel()
    nb = -(-N // block)
    if out is None:
        out = (torch.empty(B, nb, dtype=torch.uint8, device=region.device),
               torch.empty(B, nb, dtype=torch.uint8, device=region.device))
    s = Shape(B, 1, N, 64, block)
    _check(lib().carnator_region_block_flags(_ptr(region), int(n_text), ctypes.byref(s), _ptr(out[0]), _ptr(out[1]),
                                             _stream(region)))
    return out


def compact_block_mask_bits_region(bits: torch.Tensor, active_q, context_k, out=None,
                                   workspace: Optional[torch.Tensor] = None, attn=None):
    """(row_ptr, col_idx, order, n_active) of the packed mask restricted to
    active rows and context columns (carnator_compact_block_mask_bits_region).
    col_idx keeps its full capacity and n_active stays on the device (an int32
    tensor of one element), so nothing synchronises.  attn as in
    compact_block_mask."""
    B, H, nb = _bits_shape(bits)
    R = B * H * nb
    dev = bits.device
    act = _dev_u8(active_q, dev, (B, nb))
    ctx = _dev_u8(context_k, dev, (B, nb))
    s = _mask_shape(B, H, nb, attn)
    if out is None:
        out = (torch.empty(R + 1, dtype=torch.int32, device=dev),
               torch.empty(max(R * nb, 1), dtype=torch.int32, device=dev),
               torch.empty(R, dtype=torch.int32, device=dev),
               torch.empty(1, dtype=torch.int32, device=dev))
    row_ptr, col_idx, order, n_active = out
    if row_ptr.numel() < R + 1 or col_idx.numel() < R * nb or order.numel() < R or n_active.numel() < 1:
        raise ValueError("out tensors too small")
    if workspace is None:
        workspace = compact_block_mask_bits_workspace(bits)
    _check(lib().carnator_compact_block_mask_bits_region(_ptr(bits), ctypes.byref(s), _ptr(act), _ptr(ctx),
                                                         _ptr(row_ptr), _ptr(col_idx), _ptr(order), _ptr(n_active),
                                                         _ptr(workspace), workspace.numel(), _stream(bits)))
    return row_ptr, col_idx, order, n_active


def signature_sim_workspace(nq: int, m: int, topk: int, device) -> torch.Tensor:
    return _workspace(lib().carnator_signature_sim_workspace_size(nq, m, topk), device)


def signature_sim(query: torch.Tensor, bank: torch.Tensor, topk: int, return_all: bool = False,
                  workspace: Optional[torch.Tensor] = None, out=None):
    """Top-k cosine of each query row against the bank (carnator_signature_sim).

    Returns (idx int32 [nq, k], sim fp32 [nq, k]) and, with return_all, every
    cosine fp32 [nq, M].  ``out`` may pass preallocated (idx, sim).
    """
    if query.dim() == 1:
        query = query[None]
    if query.dtype != torch.float32 or bank.dtype != torch.float32 or bank.dim() != 2:
        raise ValueError("query [nq, D] and bank [M, ld] must be fp32")
    if not query.is_contiguous() or bank.stride(1) != 1:
        raise ValueError("query must be contiguous and bank rows contiguous")
    nq, dim = query.shape
    m = bank.shape[0]
    dev = query.device
    if out is not None:
        idx, sim = out
    else:
        idx = torch.empty(nq, topk, dtype=torch.int32, device=dev)
        sim = torch.empty(nq, topk, dtype=torch.float32, device=dev)
    allsim = torch.empty(nq, m, dtype=torch.float32, device=dev) if return_all else None
    L = lib()
    if workspace is None:
        workspace = signature_sim_workspace(nq, m, topk, dev)
    _check(L.carnator_signature_sim(_ptr(query), nq, _ptr(bank), m, dim, bank.stride(0), int(topk), _ptr(idx),
                                    _ptr(sim), _ptr(allsim), _ptr(workspace), workspace.numel(), _stream(query)))
    return (idx, sim, allsim) if return_all else (idx, sim)


def signature_sim_noalloc(query: torch.Tensor, bank: torch.Tensor, topk: int, return_all: bool = False,
                          out=None):
    """signature_sim on the library's own scratch (carnator_signature_sim_noalloc):
    no workspace is allocated by the call.  ``out`` may pass preallocated
    (idx, sim) so that the call allocates nothing at all."""
    if query.dim() == 1:
        query = query[None]
    if query.dtype != torch.float32 or bank.dtype != torch.float32 or bank.dim() != 2:
        raise ValueError("query [nq, D] and bank [M, ld] must be fp32")
    if not query.is_contiguous() or bank.stride(1) != 1:
        raise ValueError("query must be contiguous and bank rows contiguous")
    nq, dim = query.shape
    m = bank.shape[0]
    dev = query.device
    if out is not None:
        idx, sim = out
    else:
        idx = torch.empty(nq, topk, dtype=torch.int32, device=dev)
        sim = torch.empty(nq, topk, dtype=torch.float32, device=dev)
    allsim = torch.empty(nq, m, dtype=torch.float32, device=dev) if return_all else None
    _check(lib().carnator_signature_sim_noalloc(_ptr(query), nq, _ptr(bank), m, dim, bank.stride(0), int(topk),
                                                _ptr(idx), _ptr(sim), _ptr(allsim), _stream(query)))
    return (idx, sim, allsim) if return_all else (idx, sim)


# ---------------------------------------------------------------- compatibility gate (host)
#
# Host code on NumPy arrays: a handful of objects and candidates per request.

def _host(a, dtype, shape=None):
    import numpy as np
    a = np.ascontiguousarray(a, dtype=dtype)
    if shape is not None and a.shape != tuple(shape):
        raise ValueError("expected shape %s, got %s" % (tuple(shape), a.shape))
    return a


def _hp(a):
    return ctypes.c_void_p(a.ctypes.data)


def ciede2000(lab1, lab2):
    """CIEDE2000 of [..., 3] CIELAB arrays (carnator_ciede2000)."""
    import numpy as np
    a = _host(lab1, np.float64)
    b = _host(lab2, np.float64)
    if a.shape != b.shape or a.shape[-1] != 3:
        raise ValueError("lab1 and lab2 must have the same [..., 3] shape")
    out = np.empty(a.shape[:-1], dtype=np.float64)
    _check(lib().carnator_ciede2000(_hp(a), _hp(b), out.size, _hp(out)))
    return out


def shape_descriptor(mask, res: int = 32):
    """(area, normalised shape uint8 [res, res]) of a binary tail-frame mask
    (carnator_shape_descriptor)."""
    import numpy as np
    m = _host(np.asarray(mask) != 0, np.uint8)
    if m.ndim != 2:
        raise ValueError("mask must be [H, W]")
    area = np.zeros(1, dtype=np.float64)
    shape = np.zeros((res, res), dtype=np.uint8)
    _check(lib().carnator_shape_descriptor(_hp(m), m.shape[0], m.shape[1], res, _hp(area), _hp(shape)))
    return float(area[0]), shape


def object_discrepancy(area_q, area_j, shape_q, shape_j, lab_q, lab_j):
    """(d_size, d_shape, d_color) of one object (carnator_object_discrepancy)."""
    import numpy as np
    sq = _host(shape_q, np.uint8)
    sj = _host(shape_j, np.uint8, sq.shape)
    lq = _host(lab_q, np.float64, (3,))
    lj = _host(lab_j, np.float64, (3,))
    d = np.zeros(3, dtype=np.float64)
    _check(lib().carnator_object_discrepancy(float(area_q), float(area_j), _hp(sq), _hp(sj), sq.shape[0], _hp(lq),
                                             _hp(lj), _hp(d)))
    return d


def compat_gate(d_candidates, tau) -> int:
    """First candidate (recall order) with every discrepancy within its
    threshold, or -1 (carnator_compat_gate)."""
    import numpy as np
    d = _host(d_candidates, np.float64)
    t = _host(tau, np.float64)
    if d.ndim != 2 or d.shape[1] != t.size:
        raise ValueError("d must be [n_candidates, len(tau)]")
    chosen = np.zeros(1, dtype=np.int32)
    _check(lib().carnator_compat_gate(_hp(d), d.shape[0], t.size, _hp(t), _hp(chosen)))
    return int(chosen[0])


def clopper_pearson_upper(u: int, n: int, alpha: float) -> float:
    """One-sided Clopper-Pearson upper bound (carnator_clopper_pearson_upper)."""
    import numpy as np
    out = np.zeros(1, dtype=np.float64)
    _check(lib().carnator_clopper_pearson_upper(int(u), int(n), float(alpha), _hp(out)))
    return float(out[0])
