"""ctypes binding of libekv (argument marshalling only).

Every function here forwards to the C ABI declared in ``include/ekv.h``;
all computation happens in the library's HIP kernels.  Device arrays are
passed as torch CUDA tensors (torch is used for device memory and streams
only); host mirrors as NumPy arrays.  A missing or unbuilt library raises
``EkvError`` -- there is no fallback path.
"""

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libekv.so")

OK, ERR_INVALID, ERR_UNSUPPORTED, ERR_HIP, ERR_HOST = 0, 1, 2, 3, 4
DTYPE_BF16, DTYPE_FP16, DTYPE_FP32, DTYPE_E5M2 = 0, 1, 2, 3
MODE_NATIVE, MODE_STRUCTURED, MODE_GENERAL = 0, 1, 2
HEAD_DIM, PAGE = 128, 16


class EkvError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"ekv status {status}: {msg}")
        self.status = status


class Pool(ctypes.Structure):
    _fields_ = [("kv", ctypes.c_void_p), ("num_blocks", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class Batch(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("max_blocks", ctypes.c_int32), ("mode", ctypes.c_int32),
                ("max_seq_len", ctypes.c_int32), ("seq_lens", ctypes.c_void_p),
                ("block_table", ctypes.c_void_p), ("tags", ctypes.c_void_p),
                ("boundaries", ctypes.c_void_p)]


class CtrlConfig(ctypes.Structure):
    _fields_ = [("min_batch", ctypes.c_int32), ("decay", ctypes.c_int32), ("a_max", ctypes.c_int32),
                ("sink_pairs", ctypes.c_int32), ("recent_pairs", ctypes.c_int32), ("policy", ctypes.c_int32),
                ("watermark", ctypes.c_int32), ("flags", ctypes.c_int32)]


class CtrlState(ctypes.Structure):
    _fields_ = [("reserve", ctypes.c_int32), ("surplus", ctypes.c_int32), ("shortage", ctypes.c_int32),
                ("budget", ctypes.c_int32)]


CTRL_SHORTAGE, CTRL_WATERMARK = 0, 1

# violation kinds of the device-side checks, in the order of EKV_VIOL_*
VIOLATIONS = ("seq_len", "block_range", "tag_value", "pair_mixed", "base_partial", "base_alias", "mode",
              "list_range", "list_state", "list_partial", "list_duplicate", "new_block")
NO_INDEX = 0x7FFFFFFF
CTRL_EAGER_PROMOTION, CTRL_NO_PROMOTION = 1, 2


# name -> (restype, argtypes), in the order of include/ekv.h
_P, _I, _U, _F, _S = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t, ctypes.c_float, ctypes.c_void_p
SIGNATURES = {
    "ekv_status_string": (ctypes.c_char_p, [_I]),
    "ekv_last_error": (ctypes.c_char_p, []),
    "ekv_version": (ctypes.c_char_p, []),
    "ekv_lower": (_I, [_P, _P, _I, _I, _I, _P, _P]),
    "ekv_decode_workspace_bytes": (_U, [ctypes.POINTER(Pool), ctypes.POINTER(Batch)]),
    "ekv_decode_workspace_init": (_I, [_P, _U, _S]),
    "ekv_attn_decode": (_I, [ctypes.POINTER(Pool), ctypes.POINTER(Batch), _P, _P, _I, _F, _P, _U, _S]),
    "ekv_attn_decode_append": (_I, [ctypes.POINTER(Pool), ctypes.POINTER(Batch), _P, _P, _P, _P, _I, _F, _P,
                                    ctypes.c_size_t, _S]),
    "ekv_attn_decode_noalloc": (_I, [ctypes.POINTER(Pool), ctypes.POINTER(Batch), _P, _P, _I, _F, _S]),
    "ekv_attn_prefill": (_I, [ctypes.POINTER(Pool), ctypes.POINTER(Batch), _P, _P, _I, _I, _P, _I, _F, _S]),
    "ekv_append_kv": (_I, [ctypes.POINTER(Pool), _P, _P, _P, _I, _S]),
    "ekv_demote": (_I, [ctypes.POINTER(Pool), _I, _P, _P, _P, _I, _I, _P, _P, _S]),
    "ekv_refine": (_I, [ctypes.POINTER(Pool), _I, _P, _P, _P, _P, _I, _I, _P, _S]),
    "ekv_refine_staged": (_I, [ctypes.POINTER(Pool), _I, _P, _P, _P, _P, _I, _I, _S]),
    "ekv_stage_blocks": (_I, [ctypes.POINTER(Pool), _I, _P, _P, _S]),
    "ekv_promote_begin": (_I, [ctypes.POINTER(Pool), _I, _P, _P, _P, _S]),
    "ekv_promote_publish": (_I, [ctypes.POINTER(Pool), _I, _P, _P, _P, _P, _I, _I, _P, _S]),
    "ekv_demote_layers": (_I, [ctypes.POINTER(Pool), _P, _I, _I, _P, _P, _P, _I, _I, _P, _P, _S]),
    "ekv_refine_layers": (_I, [ctypes.POINTER(Pool), _P, _I, _I, _P, _P, _P, _P, _I, _I, _P, _S]),
    "ekv_check_transition": (_I, [_I, _P, _I, _P, _P, _P, _I, _I, _I, _I, _P]),
    "ekv_validate_batch": (_I, [ctypes.POINTER(Pool), ctypes.POINTER(Batch), _P, _S]),
    "ekv_validate_transition": (_I, [ctypes.POINTER(Pool), _I, _I, _P, _P, _P, _P, _P, _I, _I, _P, _S]),
    "ekv_ctrl_demotion": (_I, [ctypes.POINTER(CtrlConfig), ctypes.POINTER(CtrlState), _I, _I, _P, _P, _P,
                               _I, _I, _I, _P, _I, _P]),
    "ekv_ctrl_promotion": (_I, [ctypes.POINTER(CtrlConfig), ctypes.POINTER(CtrlState), _I, _I, _P, _P, _I,
                                _I, _I, _P, _I, _P]),
}

_lib = None


def lib():
    """The loaded library; raises EkvError if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise EkvError(ERR_HIP, f"{LIB_PATH} not built (run __graft_entry__.build())")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype, fn.argtypes = res, args
        _lib = handle
    return _lib


def _check(status):
    if status != OK:
        L = lib()
        raise EkvError(status, f"{L.ekv_status_string(status).decode()}: {L.ekv_last_error().decode()}")


def _ptr(t):
    """Device pointer of a contiguous torch GPU tensor, or None.  A CPU
    tensor is refused here: its address is host memory no kernel may read
    (pinned host buffers are passed with :func:`_host_ptr`)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise EkvError(ERR_INVALID, "device argument must be a GPU tensor")
    if not t.is_contiguous():
        raise EkvError(ERR_INVALID, "tensor must be contiguous")
    return t.data_ptr()


def _host_ptr(t):
    """Address of a contiguous tensor that may also live in pinned host
    memory (the refinement bytes); the library itself checks that the
    device can read it."""
    if t is None:
        return None
    if not t.is_contiguous():
        raise EkvError(ERR_INVALID, "tensor must be contiguous")
    return t.data_ptr()


def _host(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(ctypes.c_void_p)


def _stream(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def dtype_code(torch_dtype):
    import torch
    return {torch.bfloat16: DTYPE_BF16, torch.float16: DTYPE_FP16, torch.float32: DTYPE_FP32}[torch_dtype]


def make_pool(kv, num_kv_heads, dtype_name="bf16"):
    """Describe a device pool tensor [NB][2][Hkv][16][128] of 16-bit words
    (bf16, fp16) or bytes (e5m2)."""
    nb = kv.numel() // (2 * num_kv_heads * PAGE * HEAD_DIM)
    code = {"bf16": DTYPE_BF16, "fp16": DTYPE_FP16, "e5m2": DTYPE_E5M2}[dtype_name]
    return Pool(_ptr(kv), nb, num_kv_heads, PAGE, HEAD_DIM, code)


def make_batch(seq_lens, block_table, tags, boundaries, num_q_heads, mode, max_seq_len=0):
    """Describe a batch; the tensors are device int32/uint8 arrays."""
    bsz, max_blocks = block_table.shape
    return Batch(bsz, num_q_heads, max_blocks, mode, int(max_seq_len), _ptr(seq_lens),
                 _ptr(block_table), _ptr(tags), _ptr(boundaries))


def lower(tags, seq_lens, page=PAGE):
    """Host lowering: returns (mode, boundaries int32 [B][2])."""
    tags, tp = _host(tags, np.uint8)
    seq_lens, sp = _host(seq_lens, np.int32)
    bsz, max_blocks = tags.shape
    bounds = np.zeros((bsz, 2), dtype=np.int32)
    mode = ctypes.c_int32(-1)
    _check(lib().ekv_lower(tp, sp, bsz, max_blocks, page, ctypes.byref(mode),
                           bounds.ctypes.data_as(ctypes.c_void_p)))
    return mode.value, bounds


def decode_workspace_bytes(pool, batch):
    return lib().ekv_decode_workspace_bytes(ctypes.byref(pool), ctypes.byref(batch))


def decode_workspace(pool, batch, device="cuda"):
    """A zero-filled decode workspace (its merge counters start at zero)."""
    import torch
    return torch.zeros(decode_workspace_bytes(pool, batch), dtype=torch.uint8, device=device)


def decode_workspace_init(ws, stream=None):
    _check(lib().ekv_decode_workspace_init(_ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def attn_decode(pool, batch, q, out, scale, ws, stream=None):
    _check(lib().ekv_attn_decode(ctypes.byref(pool), ctypes.byref(batch), _ptr(q), _ptr(out),
                                 dtype_code(out.dtype), scale, _ptr(ws), ws.numel() * ws.element_size(),
                                 _stream(stream)))


def attn_decode_append(pool, batch, q, k_new, v_new, out, scale, ws, stream=None):
    """Append each sequence's newest token (k_new / v_new [B][Hkv][D]) and decode, in one launch."""
    _check(lib().ekv_attn_decode_append(ctypes.byref(pool), ctypes.byref(batch), _ptr(q), _ptr(k_new), _ptr(v_new),
                                        _ptr(out), dtype_code(out.dtype), scale, _ptr(ws),
                                        ws.numel() * ws.element_size(), _stream(stream)))


def attn_decode_noalloc(pool, batch, q, out, scale, stream=None):
    """Decode on the library's static scratch (no workspace, no allocation)."""
    _check(lib().ekv_attn_decode_noalloc(ctypes.byref(pool), ctypes.byref(batch), _ptr(q), _ptr(out),
                                         dtype_code(out.dtype), scale, _stream(stream)))


def attn_prefill(pool, batch, q, cu_q, max_q_len, out, scale, stream=None):
    _check(lib().ekv_attn_prefill(ctypes.byref(pool), ctypes.byref(batch), _ptr(q), _ptr(cu_q),
                                  q.shape[0], int(max_q_len), _ptr(out), dtype_code(out.dtype), scale,
                                  _stream(stream)))


def append_kv(pool, slots, k, v, stream=None):
    _check(lib().ekv_append_kv(ctypes.byref(pool), _ptr(slots), _ptr(k), _ptr(v), slots.numel(),
                               _stream(stream)))


def demote(pool, pairs, block_table, tags, freed_out, lo_out=None, stream=None):
    bsz, max_blocks = block_table.shape
    _check(lib().ekv_demote(ctypes.byref(pool), pairs.shape[0], _ptr(pairs), _ptr(block_table),
                            _ptr(tags), bsz, max_blocks, _ptr(freed_out), _host_ptr(lo_out), _stream(stream)))


def refine(pool, pairs, new_blocks, block_table, tags, lo_in, stream=None):
    bsz, max_blocks = block_table.shape
    _check(lib().ekv_refine(ctypes.byref(pool), pairs.shape[0], _ptr(pairs), _ptr(new_blocks),
                            _ptr(block_table), _ptr(tags), bsz, max_blocks, _host_ptr(lo_in), _stream(stream)))


def refine_staged(pool, pairs, new_blocks, block_table, tags, stream=None):
    """Refinement whose bytes were copied into each pair's new block beforehand."""
    bsz, max_blocks = block_table.shape
    _check(lib().ekv_refine_staged(ctypes.byref(pool), pairs.shape[0], _ptr(pairs), _ptr(new_blocks),
                                   _ptr(block_table), _ptr(tags), bsz, max_blocks, _stream(stream)))


def stage_blocks(pool, sources, new_blocks, stream=None):
    """Copy one block's bytes from each source address (device memory or
    pinned host memory) into the blocks new_blocks (host int32 array)."""
    srcs = np.ascontiguousarray([int(a) for a in sources], dtype=np.uint64)
    new, np_ = _host(new_blocks, np.int32)
    if len(srcs) != len(new):
        raise EkvError(ERR_INVALID, "one new block per source")
    _check(lib().ekv_stage_blocks(ctypes.byref(pool), len(new), srcs.ctypes.data_as(ctypes.c_void_p), np_,
                                  _stream(stream)))


def _event(event, create_on=None):
    """The HIP event handle of a torch.cuda.Event.  torch creates the event
    at its first record; with create_on (a stream) an event not yet created
    is recorded there once first, otherwise it must exist already."""
    if event is None:
        return None
    if event.cuda_event == 0:
        if create_on is None:
            raise EkvError(ERR_INVALID, "the event has never been recorded")
        event.record(create_on)
    return ctypes.c_void_p(event.cuda_event)


def promote_begin(pool, sources, new_blocks, copied, copy_stream=None):
    """ekv_promote_begin: stage each source (pinned host or device address)
    into new_blocks (host int32 array) on copy_stream, then record the
    torch.cuda.Event `copied` there."""
    srcs = np.ascontiguousarray([int(a) for a in sources], dtype=np.uint64)
    new, np_ = _host(new_blocks, np.int32)
    if len(srcs) != len(new):
        raise EkvError(ERR_INVALID, "one new block per source")
    import torch
    cs = copy_stream if copy_stream is not None else torch.cuda.current_stream()
    _check(lib().ekv_promote_begin(ctypes.byref(pool), len(new), srcs.ctypes.data_as(ctypes.c_void_p), np_,
                                   _event(copied, cs), _stream(cs)))


def promote_publish(pool, pairs, new_blocks, block_table, tags, copied, stream=None):
    """ekv_promote_publish: `stream` waits for `copied`, then the staged
    refinement publishes the pairs (pairs, new_blocks: device tensors)."""
    bsz, max_blocks = block_table.shape
    _check(lib().ekv_promote_publish(ctypes.byref(pool), pairs.shape[0], _ptr(pairs), _ptr(new_blocks),
                                     _ptr(block_table), _ptr(tags), bsz, max_blocks, _event(copied),
                                     _stream(stream)))


def demote_layers(pool, layer_kv, pairs, block_table, tags, freed_out, lo_out=None, stream=None):
    """layer_kv: device int64 tensor [L] of the layers' pool addresses."""
    bsz, max_blocks = block_table.shape
    _check(lib().ekv_demote_layers(ctypes.byref(pool), _ptr(layer_kv), layer_kv.shape[0], pairs.shape[0],
                                   _ptr(pairs), _ptr(block_table), _ptr(tags), bsz, max_blocks, _ptr(freed_out),
                                   _host_ptr(lo_out), _stream(stream)))


def refine_layers(pool, layer_kv, pairs, new_blocks, block_table, tags, lo_in, stream=None):
    bsz, max_blocks = block_table.shape
    _check(lib().ekv_refine_layers(ctypes.byref(pool), _ptr(layer_kv), layer_kv.shape[0], pairs.shape[0],
                                   _ptr(pairs), _ptr(new_blocks), _ptr(block_table), _ptr(tags), bsz, max_blocks,
                                   _host_ptr(lo_in), _stream(stream)))


def check_transition(kind, pairs, block_table, tags, seq_lens, num_blocks, new_blocks=None, page=PAGE):
    """Host validation of a demotion (kind 0) or refinement (kind 1) list.
    Returns (ok: bool, message: str)."""
    pairs, pp = _host(np.asarray(pairs).reshape(-1, 2), np.int32)
    bt, bp = _host(block_table, np.int32)
    tg, tgp = _host(tags, np.uint8)
    sl, sp = _host(seq_lens, np.int32)
    nbp = None
    if new_blocks is not None:
        nbk, nbp = _host(new_blocks, np.int32)
    status = lib().ekv_check_transition(kind, pp, pairs.shape[0], bp, tgp, sp, bt.shape[0],
                                        bt.shape[1], page, num_blocks, nbp)
    return status == OK, (lib().ekv_last_error().decode() if status != OK else "")


def _read_report(report, stream):
    import torch
    if stream is not None:
        stream.synchronize()
    else:
        torch.cuda.current_stream().synchronize()
    h = report.cpu().numpy()
    n = len(VIOLATIONS)
    return {name: (int(h[k]), int(h[n + k])) for k, name in enumerate(VIOLATIONS)}


def validate_batch(pool, batch, stream=None):
    """Device-side check of a batch's metadata.  Returns {kind: (count,
    smallest index)} (index NO_INDEX when the count is 0); synchronises."""
    import torch
    report = torch.empty(2 * len(VIOLATIONS), dtype=torch.int32, device="cuda")
    _check(lib().ekv_validate_batch(ctypes.byref(pool), ctypes.byref(batch), _ptr(report), _stream(stream)))
    return _read_report(report, stream)


def validate_transition(pool, kind, pairs, block_table, tags, seq_lens=None, new_blocks=None, stream=None):
    """Device-side check of a demotion (kind 0) or refinement (kind 1) list;
    as validate_batch."""
    import torch
    report = torch.empty(2 * len(VIOLATIONS), dtype=torch.int32, device="cuda")
    bsz, max_blocks = block_table.shape
    _check(lib().ekv_validate_transition(ctypes.byref(pool), kind, pairs.shape[0], _ptr(pairs), _ptr(new_blocks),
                                         _ptr(block_table), _ptr(tags), _ptr(seq_lens), bsz, max_blocks,
                                         _ptr(report), _stream(stream)))
    return _read_report(report, stream)


def ctrl_config(min_batch=16, decay=2, a_max=-1, sink_pairs=0, recent_pairs=0, policy=CTRL_SHORTAGE,
                watermark=0, eager=False, no_promotion=False):
    """Controller parameters (defaults: App. B.1's B_min = 16, lambda = 2)."""
    flags = (CTRL_EAGER_PROMOTION if eager else 0) | (CTRL_NO_PROMOTION if no_promotion else 0)
    return CtrlConfig(min_batch, decay, a_max, sink_pairs, recent_pairs, policy, watermark, flags)


def ctrl_demotion(cfg, state, demand, free, tags, seq_lens, backed=None, page=PAGE):
    """First half of a control step: returns the pairs to demote (int32 [n][2])."""
    tags, tp = _host(tags, np.uint8)
    seq_lens, sp = _host(seq_lens, np.int32)
    bkp = None
    if backed is not None:
        backed, bkp = _host(backed, np.uint8)
    bsz, max_blocks = tags.shape
    cap = bsz * (max_blocks // 2)
    out = np.zeros((max(cap, 1), 2), dtype=np.int32)
    n = ctypes.c_int32(0)
    _check(lib().ekv_ctrl_demotion(ctypes.byref(cfg), ctypes.byref(state), int(demand), int(free), tp, sp, bkp,
                                   bsz, max_blocks, page, out.ctypes.data_as(ctypes.c_void_p), cap,
                                   ctypes.byref(n)))
    return out[:n.value].copy()


def ctrl_promotion(cfg, state, free_post, slack, tags, seq_lens, page=PAGE):
    """Second half, after scheduling: returns the pairs to promote (int32 [n][2])."""
    tags, tp = _host(tags, np.uint8)
    seq_lens, sp = _host(seq_lens, np.int32)
    bsz, max_blocks = tags.shape
    cap = bsz * (max_blocks // 2)
    out = np.zeros((max(cap, 1), 2), dtype=np.int32)
    n = ctypes.c_int32(0)
    _check(lib().ekv_ctrl_promotion(ctypes.byref(cfg), ctypes.byref(state), int(free_post), int(slack), tp, sp,
                                    bsz, max_blocks, page, out.ctypes.data_as(ctypes.c_void_p), cap,
                                    ctypes.byref(n)))
    return out[:n.value].copy()
