"""Thin Python binding of the chunked verification-attention C-ABI.

Argument marshalling only: every step of the computation runs in the HIP
kernels of ``libspecmoe_verify.so``; PyTorch supplies device memory and the
stream.  There is no fallback path: if the shared library is missing, every
entry point raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

LIB_NAME = "libspecmoe_verify.so"
LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), LIB_NAME)

SPECMOE_F32 = 0
SPECMOE_BF16 = 1
SPECMOE_F16 = 2

STATUS = {
    0: "SPECMOE_OK", -1: "SPECMOE_ERR_NULL_POINTER", -2: "SPECMOE_ERR_SHAPE", -3: "SPECMOE_ERR_GQA",
    -4: "SPECMOE_ERR_HEAD_DIM", -5: "SPECMOE_ERR_DTYPE", -6: "SPECMOE_ERR_ROWS", -7: "SPECMOE_ERR_GRID",
    -8: "SPECMOE_ERR_WORKSPACE", -9: "SPECMOE_ERR_ALIGN", -10: "SPECMOE_ERR_SCALE", -11: "SPECMOE_ERR_LAUNCH",
    -12: "SPECMOE_ERR_FLAGS", -13: "SPECMOE_ERR_MASK", -14: "SPECMOE_ERR_PAGES", -15: "SPECMOE_ERR_HANDOFF",
}
SPECMOE_FLAG_NO_WAIT = 1


class Desc(ctypes.Structure):
    """Mirror of ``specmoe_verify_desc``."""
    _fields_ = [
        ("B", ctypes.c_int32), ("Hq", ctypes.c_int32), ("Hkv", ctypes.c_int32), ("D", ctypes.c_int32),
        ("C_max", ctypes.c_int32), ("S_max", ctypes.c_int32), ("dtype", ctypes.c_int32),
        ("grid_blocks", ctypes.c_int32), ("flags", ctypes.c_int32),
        ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t),
    ]


class AcceptDesc(ctypes.Structure):
    """Mirror of ``specmoe_accept_desc``."""
    _fields_ = [
        ("B", ctypes.c_int32), ("C_max", ctypes.c_int32), ("V", ctypes.c_int32), ("dtype", ctypes.c_int32),
        ("split", ctypes.c_int32), ("flags", ctypes.c_int32),
        ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t),
    ]


class PagedKV(ctypes.Structure):
    """Mirror of ``specmoe_paged_kv``."""
    _fields_ = [("page_size", ctypes.c_int32), ("pages_per_seq", ctypes.c_int32), ("num_pages", ctypes.c_int32)]


class SpecMoEError(RuntimeError):
    def __init__(self, status: int, text: str):
        super().__init__(f"{STATUS.get(status, status)}: {text}")
        self.status = status


_lib = None


def load_library(path: Optional[str] = None) -> ctypes.CDLL:
    """Load the HIP library (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(
            f"{p} is missing: build the HIP library first (python paper_2508_21706_amd/build.py)")
    lib = ctypes.CDLL(p)
    lib.specmoe_verify_attn.restype = ctypes.c_int
    lib.specmoe_verify_attn.argtypes = [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(Desc)]
    lib.specmoe_verify_attn_noalloc.restype = ctypes.c_int
    lib.specmoe_verify_attn_noalloc.argtypes = lib.specmoe_verify_attn.argtypes
    lib.specmoe_verify_attn_tree.restype = ctypes.c_int
    lib.specmoe_verify_attn_tree.argtypes = [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(Desc)]
    lib.specmoe_verify_attn_paged.restype = ctypes.c_int
    lib.specmoe_verify_attn_paged.argtypes = [ctypes.c_void_p] * 7 + [
        ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(Desc), ctypes.POINTER(PagedKV)]
    lib.specmoe_verify_attn_workspace_bytes.restype = ctypes.c_size_t
    lib.specmoe_verify_attn_workspace_bytes.argtypes = [ctypes.POINTER(Desc)]
    lib.specmoe_verify_attn_workspace_init.restype = ctypes.c_int
    lib.specmoe_verify_attn_workspace_init.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                                       ctypes.POINTER(Desc)]
    lib.specmoe_verify_attn_status.restype = ctypes.c_int
    lib.specmoe_verify_attn_status.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    lib.specmoe_verify_attn_key_tile.restype = ctypes.c_int32
    lib.specmoe_verify_attn_key_tile.argtypes = [ctypes.POINTER(Desc)]
    lib.specmoe_accept_greedy.restype = ctypes.c_int
    lib.specmoe_accept_greedy.argtypes = [ctypes.c_void_p] * 9 + [ctypes.POINTER(AcceptDesc)]
    lib.specmoe_accept_greedy_tree.restype = ctypes.c_int
    lib.specmoe_accept_greedy_tree.argtypes = [ctypes.c_void_p] * 11 + [ctypes.POINTER(AcceptDesc)]
    lib.specmoe_compact_accepted_kv.restype = ctypes.c_int
    lib.specmoe_compact_accepted_kv.argtypes = [ctypes.c_void_p] * 5 + [ctypes.POINTER(Desc)]
    lib.specmoe_accept_workspace_bytes.restype = ctypes.c_size_t
    lib.specmoe_accept_workspace_bytes.argtypes = [ctypes.POINTER(AcceptDesc)]
    lib.specmoe_accept_workspace_init.restype = ctypes.c_int
    lib.specmoe_accept_workspace_init.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                                  ctypes.POINTER(AcceptDesc)]
    lib.specmoe_status_str.restype = ctypes.c_char_p
    lib.specmoe_status_str.argtypes = [ctypes.c_int]
    if path is None:
        _lib = lib
    return lib


def status_str(status: int) -> str:
    return load_library().specmoe_status_str(status).decode()


def make_desc(B, Hq, Hkv, D, C_max, S_max, dtype: int, grid_blocks: int = 0, flags: int = 0,
              workspace: Optional[torch.Tensor] = None) -> Desc:
    d = Desc(B, Hq, Hkv, D, C_max, S_max, dtype, grid_blocks, flags, None, 0)
    if workspace is not None:
        d.workspace = workspace.data_ptr()
        d.workspace_bytes = workspace.numel() * workspace.element_size()
    return d


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return SPECMOE_BF16
    if t.dtype == torch.float16:
        return SPECMOE_F16
    if t.dtype == torch.float32:
        return SPECMOE_F32
    raise TypeError(f"unsupported dtype {t.dtype}; expected torch.bfloat16, torch.float16 or torch.float32")


def desc_for(q: torch.Tensor, k_cache: torch.Tensor, grid_blocks: int = 0) -> Desc:
    B, C_max, Hq, D = q.shape
    _, Hkv, S_max, _ = k_cache.shape
    return make_desc(B, Hq, Hkv, D, C_max, S_max, _dtype_code(q), grid_blocks)


def workspace_bytes(desc: Desc) -> int:
    return int(load_library().specmoe_verify_attn_workspace_bytes(ctypes.byref(desc)))


def key_tile(desc: Desc) -> int:
    return int(load_library().specmoe_verify_attn_key_tile(ctypes.byref(desc)))


def alloc_workspace(desc: Desc, device, stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """Allocate a workspace for ``desc`` and zero its status word and counters
    on the stream.  The memory comes from the stream's own pool of the caching
    allocator, so that when the tensor is dropped, the block is only reused by
    work ordered after what was enqueued on that stream."""
    n = workspace_bytes(desc)
    if n == 0:
        raise SpecMoEError(-2, "invalid descriptor")
    s = stream if stream is not None else torch.cuda.current_stream(device)
    with torch.cuda.stream(s):
        ws = torch.empty(n, dtype=torch.uint8, device=device)
    st = load_library().specmoe_verify_attn_workspace_init(ws.data_ptr(), n, s.cuda_stream, ctypes.byref(desc))
    if st != 0:
        raise SpecMoEError(st, status_str(st))
    return ws


def workspace_status(workspace: Optional[torch.Tensor], stream: Optional[torch.cuda.Stream] = None) -> int:
    """``specmoe_verify_attn_status``: synchronises with the stream and returns
    0 (SPECMOE_OK) or -15 (SPECMOE_ERR_HANDOFF: an in-kernel wait gave up in a
    call since the workspace was initialised).  ``workspace=None``: the
    current device's static scratch of ``verify_attn_noalloc``."""
    if workspace is None:
        s = stream if stream is not None else torch.cuda.current_stream()
        st = load_library().specmoe_verify_attn_status(None, 0, s.cuda_stream)
    else:
        s = stream if stream is not None else torch.cuda.current_stream(workspace.device)
        st = load_library().specmoe_verify_attn_status(workspace.data_ptr(),
                                                        workspace.numel() * workspace.element_size(), s.cuda_stream)
    if st not in (0, -15):
        raise SpecMoEError(st, status_str(st))
    return st


def _check(t: torch.Tensor, name: str, shape, dtype):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.dtype != dtype:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def verify_attn(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                ctx_lens: torch.Tensor, chunk_lens: torch.Tensor, scale: float,
                out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                workspace: Optional[torch.Tensor] = None, grid_blocks: int = 0,
                stream: Optional[torch.cuda.Stream] = None, flags: int = 0,
                check_lengths: bool = False):
    """Chunked verification attention; see ``include/specmoe_verify.h``.

    q [B, C_max, Hq, D], k_cache / v_cache [B, Hkv, S_max, D] (bf16, f16 or f32),
    ctx_lens / chunk_lens int32 [B], all on the GPU.  Returns (out, lse) as
    float32 [B, C_max, Hq, D] and [B, C_max, Hq].  ``workspace`` (from
    ``alloc_workspace``) is reused across calls; without one, a fresh
    workspace is allocated and zeroed.  ``check_lengths`` copies the
    lengths to the host (a synchronisation) and checks the kernel's
    preconditions; off by default.  Repeated calls with the same inputs and
    grid give bitwise-identical results.
    """
    return _call(q, k_cache, v_cache, ctx_lens, chunk_lens, None, scale, out, lse, workspace, grid_blocks,
                 stream, flags, check_lengths)


def verify_attn_noalloc(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                        ctx_lens: torch.Tensor, chunk_lens: torch.Tensor, scale: float,
                        out: torch.Tensor, lse: torch.Tensor, grid_blocks: int = 0,
                        stream: Optional[torch.cuda.Stream] = None):
    """``specmoe_verify_attn_noalloc``: chain drafts like ``verify_attn``,
    with the library's static per-GPU scratch instead of a workspace.  The
    caller passes ``out`` and ``lse``; nothing is allocated.  Calls that may
    overlap on one GPU race (they share the scratch)."""
    lib = load_library()
    B, C_max, Hq, D = q.shape
    if k_cache.dim() != 4:
        raise ValueError("k_cache must be [B, Hkv, S_max, D]")
    _, Hkv, S_max, _ = k_cache.shape
    dt = q.dtype
    _check(q, "q", (B, C_max, Hq, D), dt)
    _check(k_cache, "k_cache", (B, Hkv, S_max, D), dt)
    _check(v_cache, "v_cache", (B, Hkv, S_max, D), dt)
    _check(ctx_lens, "ctx_lens", (B,), torch.int32)
    _check(chunk_lens, "chunk_lens", (B,), torch.int32)
    _check(out, "out", (B, C_max, Hq, D), torch.float32)
    _check(lse, "lse", (B, C_max, Hq), torch.float32)
    desc = make_desc(B, Hq, Hkv, D, C_max, S_max, _dtype_code(q), grid_blocks)
    s = stream if stream is not None else torch.cuda.current_stream(q.device)
    st = lib.specmoe_verify_attn_noalloc(q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), ctx_lens.data_ptr(),
                                         chunk_lens.data_ptr(), float(scale), out.data_ptr(), lse.data_ptr(),
                                         s.cuda_stream, ctypes.byref(desc))
    if st != 0:
        raise SpecMoEError(st, status_str(st))
    return out, lse


def verify_attn_tree(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                     ctx_lens: torch.Tensor, chunk_lens: torch.Tensor, draft_mask: torch.Tensor, scale: float,
                     out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                     workspace: Optional[torch.Tensor] = None, grid_blocks: int = 0,
                     stream: Optional[torch.cuda.Stream] = None, flags: int = 0,
                     check_lengths: bool = False):
    """Chunked verification attention for tree drafts; see
    ``specmoe_verify_attn_tree`` in ``include/specmoe_verify.h``.

    Arguments as ``verify_attn``, plus ``draft_mask``: int64 (or uint64)
    [B, C_max] on the GPU, the 64-bit draft-mask words (bit k of word
    [b, i] set: draft token i of sequence b attends to draft token k).
    C_max must be <= 64.
    """
    return _call(q, k_cache, v_cache, ctx_lens, chunk_lens, draft_mask, scale, out, lse, workspace,
                 grid_blocks, stream, flags, check_lengths)


def verify_attn_paged(q: torch.Tensor, k_pages: torch.Tensor, v_pages: torch.Tensor, block_table: torch.Tensor,
                      ctx_lens: torch.Tensor, chunk_lens: torch.Tensor, scale: float,
                      draft_mask: Optional[torch.Tensor] = None,
                      out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                      workspace: Optional[torch.Tensor] = None, grid_blocks: int = 0,
                      stream: Optional[torch.cuda.Stream] = None, flags: int = 0,
                      check_lengths: bool = False):
    """Chunked verification attention over a paged KV cache; see
    ``specmoe_verify_attn_paged`` in ``include/specmoe_verify.h``.

    k_pages / v_pages [num_pages, Hkv, page_size, D], block_table int32
    [B, pages_per_seq] (S_max = page_size * pages_per_seq); the other
    arguments as ``verify_attn`` (``draft_mask``: tree drafts, as
    ``verify_attn_tree``).
    """
    if k_pages.dim() != 4:
        raise ValueError("k_pages must be [num_pages, Hkv, page_size, D]")
    num_pages, _, page_size, _ = k_pages.shape
    if block_table.dim() != 2:
        raise ValueError("block_table must be [B, pages_per_seq]")
    _check(block_table, "block_table", (q.shape[0], block_table.shape[1]), torch.int32)
    paged = PagedKV(page_size, block_table.shape[1], num_pages)
    return _call(q, k_pages, v_pages, ctx_lens, chunk_lens, draft_mask, scale, out, lse, workspace, grid_blocks,
                 stream, flags, check_lengths, paged=paged, block_table=block_table)


def _call(q, k_cache, v_cache, ctx_lens, chunk_lens, draft_mask, scale, out, lse, workspace, grid_blocks,
          stream, flags, check_lengths, paged: Optional[PagedKV] = None, block_table=None):
    lib = load_library()
    B, C_max, Hq, D = q.shape
    if k_cache.dim() != 4:
        raise ValueError("k_cache must be [B, Hkv, S_max, D]")
    dt = q.dtype
    _check(q, "q", (B, C_max, Hq, D), dt)
    if paged is None:
        _, Hkv, S_max, _ = k_cache.shape
        _check(k_cache, "k_cache", (B, Hkv, S_max, D), dt)
        _check(v_cache, "v_cache", (B, Hkv, S_max, D), dt)
    else:
        Hkv = k_cache.shape[1]
        S_max = paged.page_size * paged.pages_per_seq
        _check(k_cache, "k_pages", (paged.num_pages, Hkv, paged.page_size, D), dt)
        _check(v_cache, "v_pages", (paged.num_pages, Hkv, paged.page_size, D), dt)
    _check(ctx_lens, "ctx_lens", (B,), torch.int32)
    _check(chunk_lens, "chunk_lens", (B,), torch.int32)
    if draft_mask is not None:
        mdt = draft_mask.dtype if draft_mask.dtype in (torch.int64, torch.uint64) else torch.int64
        _check(draft_mask, "draft_mask", (B, C_max), mdt)
    if check_lengths:
        c = chunk_lens.cpu()
        l = ctx_lens.cpu()
        if (c < 0).any() or (c > C_max).any() or (l < 0).any() or (l + c > S_max).any():
            raise ValueError("lengths break 0 <= c_b <= C_max, l_b >= 0, l_b + c_b <= S_max")
    s = stream if stream is not None else torch.cuda.current_stream(q.device)
    with torch.cuda.stream(s):   # outputs from the launch stream's pool
        if out is None:
            out = torch.empty((B, C_max, Hq, D), dtype=torch.float32, device=q.device)
        if lse is None:
            lse = torch.empty((B, C_max, Hq), dtype=torch.float32, device=q.device)
    _check(out, "out", (B, C_max, Hq, D), torch.float32)
    _check(lse, "lse", (B, C_max, Hq), torch.float32)
    desc = make_desc(B, Hq, Hkv, D, C_max, S_max, _dtype_code(q), grid_blocks, flags)
    if B == 0:
        return out, lse
    if workspace is None:
        workspace = alloc_workspace(desc, q.device, s)
    desc.workspace = workspace.data_ptr()
    desc.workspace_bytes = workspace.numel() * workspace.element_size()
    if paged is not None:
        st = lib.specmoe_verify_attn_paged(q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
                                           block_table.data_ptr(), ctx_lens.data_ptr(), chunk_lens.data_ptr(),
                                           draft_mask.data_ptr() if draft_mask is not None else None,
                                           float(scale), out.data_ptr(), lse.data_ptr(), s.cuda_stream,
                                           ctypes.byref(desc), ctypes.byref(paged))
    elif draft_mask is None:
        st = lib.specmoe_verify_attn(q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
                                     ctx_lens.data_ptr(), chunk_lens.data_ptr(), float(scale),
                                     out.data_ptr(), lse.data_ptr(), s.cuda_stream, ctypes.byref(desc))
    else:
        st = lib.specmoe_verify_attn_tree(q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
                                          ctx_lens.data_ptr(), chunk_lens.data_ptr(), draft_mask.data_ptr(),
                                          float(scale), out.data_ptr(), lse.data_ptr(), s.cuda_stream,
                                          ctypes.byref(desc))
    if st != 0:
        raise SpecMoEError(st, status_str(st))
    return out, lse


# ------------------------------------------------------------ acceptance step

def accept_desc(B, C_max, V, dtype: int, split: int = 0) -> AcceptDesc:
    return AcceptDesc(B, C_max, V, dtype, split, 0, None, 0)


def alloc_accept_workspace(desc: AcceptDesc, device, stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """Allocate a workspace for ``desc`` and zero its counters on the stream."""
    lib = load_library()
    n = int(lib.specmoe_accept_workspace_bytes(ctypes.byref(desc)))
    if n == 0:
        raise SpecMoEError(-2, "invalid acceptance descriptor")
    s = stream if stream is not None else torch.cuda.current_stream(device)
    with torch.cuda.stream(s):   # from the stream's pool (see alloc_workspace)
        ws = torch.empty(n, dtype=torch.uint8, device=device)
    st = lib.specmoe_accept_workspace_init(ws.data_ptr(), n, s.cuda_stream, ctypes.byref(desc))
    if st != 0:
        raise SpecMoEError(st, status_str(st))
    return ws


def accept_greedy_tree(logits: torch.Tensor, tokens: torch.Tensor, draft_mask: torch.Tensor, ctx_lens: torch.Tensor,
                       chunk_lens: torch.Tensor, out: Optional[dict] = None, workspace: Optional[torch.Tensor] = None,
                       split: int = 0, stream: Optional[torch.cuda.Stream] = None, in_place: bool = False):
    """Greedy acceptance of tree drafts; see ``specmoe_accept_greedy_tree``
    in ``include/specmoe_accept.h``.  As ``accept_greedy`` plus ``draft_mask``
    (int64 [B, C_max] root-path words, C_max <= 64); the result also holds
    ``path`` (int64 [B]: the accepted path's node bits).  Call
    ``compact_accepted_kv`` with the context lengths from before the step to
    move the path's K/V rows into place."""
    B, C_max = tokens.shape
    mdt = draft_mask.dtype if draft_mask.dtype in (torch.int64, torch.uint64) else torch.int64
    _check(draft_mask, "draft_mask", (B, C_max), mdt)
    if out is None:
        out = {}
    if "path" not in out:
        out["path"] = torch.empty((B,), dtype=torch.int64, device=logits.device)
    _check(out["path"], "path", (B,), torch.int64)
    return accept_greedy(logits, tokens, ctx_lens, chunk_lens, out=out, workspace=workspace, split=split,
                         stream=stream, in_place=in_place, _tree=(draft_mask, out["path"]))


def compact_accepted_kv(k_cache: torch.Tensor, v_cache: torch.Tensor, ctx_lens: torch.Tensor, path: torch.Tensor,
                        stream: Optional[torch.cuda.Stream] = None):
    """Move each sequence's accepted tree path's K/V rows to the rows right
    after its context (``specmoe_compact_accepted_kv``); ``ctx_lens`` are the
    lengths from before the acceptance step."""
    lib = load_library()
    B, Hkv, S_max, D = k_cache.shape
    _check(k_cache, "k_cache", (B, Hkv, S_max, D), k_cache.dtype)
    _check(v_cache, "v_cache", (B, Hkv, S_max, D), k_cache.dtype)
    _check(ctx_lens, "ctx_lens", (B,), torch.int32)
    _check(path, "path", (B,), path.dtype if path.dtype in (torch.int64, torch.uint64) else torch.int64)
    desc = make_desc(B, Hkv, Hkv, D, 1, S_max, _dtype_code(k_cache))
    s = stream if stream is not None else torch.cuda.current_stream(k_cache.device)
    st = lib.specmoe_compact_accepted_kv(k_cache.data_ptr(), v_cache.data_ptr(), ctx_lens.data_ptr(), path.data_ptr(),
                                         s.cuda_stream, ctypes.byref(desc))
    if st != 0:
        raise SpecMoEError(st, status_str(st))


def accept_greedy(logits: torch.Tensor, tokens: torch.Tensor, ctx_lens: torch.Tensor, chunk_lens: torch.Tensor,
                  out: Optional[dict] = None, workspace: Optional[torch.Tensor] = None, split: int = 0,
                  stream: Optional[torch.cuda.Stream] = None, in_place: bool = False, _tree=None):
    """Greedy acceptance after verification; see ``include/specmoe_accept.h``.

    logits [B, C_max, V] (bf16 or f32), tokens int32 [B, C_max], ctx_lens /
    chunk_lens int32 [B], all on the GPU.  Returns a dict of int32 tensors:
    argmax [B, C_max], accepted [B], next_token [B], new_ctx_lens [B] (with
    ``in_place``, ctx_lens itself is updated and returned as new_ctx_lens).
    ``out`` may supply those tensors.
    """
    lib = load_library()
    if logits.dim() != 3:
        raise ValueError("logits must be [B, C_max, V]")
    B, C_max, V = logits.shape
    _check(logits, "logits", (B, C_max, V), logits.dtype)
    _check(tokens, "tokens", (B, C_max), torch.int32)
    _check(ctx_lens, "ctx_lens", (B,), torch.int32)
    _check(chunk_lens, "chunk_lens", (B,), torch.int32)
    dev = logits.device
    if out is None:
        out = {}
    for key, shape in (("argmax", (B, C_max)), ("accepted", (B,)), ("next_token", (B,))):
        if key not in out:
            out[key] = torch.empty(shape, dtype=torch.int32, device=dev)
    if not in_place and "new_ctx_lens" not in out:
        out["new_ctx_lens"] = torch.empty((B,), dtype=torch.int32, device=dev)
    if in_place:
        out["new_ctx_lens"] = ctx_lens
    _check(out["argmax"], "argmax", (B, C_max), torch.int32)
    for k in ("accepted", "next_token", "new_ctx_lens"):
        _check(out[k], k, (B,), torch.int32)
    desc = accept_desc(B, C_max, V, _dtype_code(logits), split)
    s = stream if stream is not None else torch.cuda.current_stream(dev)
    if B == 0:
        return out
    if workspace is None:
        workspace = alloc_accept_workspace(desc, dev, s)
    desc.workspace = workspace.data_ptr()
    desc.workspace_bytes = workspace.numel() * workspace.element_size()
    if _tree is None:
        st = lib.specmoe_accept_greedy(logits.data_ptr(), tokens.data_ptr(), ctx_lens.data_ptr(),
                                       chunk_lens.data_ptr(), out["argmax"].data_ptr(), out["accepted"].data_ptr(),
                                       out["next_token"].data_ptr(), out["new_ctx_lens"].data_ptr(), s.cuda_stream,
                                       ctypes.byref(desc))
    else:
        st = lib.specmoe_accept_greedy_tree(logits.data_ptr(), tokens.data_ptr(), _tree[0].data_ptr(),
                                            ctx_lens.data_ptr(), chunk_lens.data_ptr(), out["argmax"].data_ptr(),
                                            out["accepted"].data_ptr(), out["next_token"].data_ptr(),
                                            out["new_ctx_lens"].data_ptr(), _tree[1].data_ptr(), s.cuda_stream,
                                            ctypes.byref(desc))
    if st != 0:
        raise SpecMoEError(st, status_str(st))
    return out
