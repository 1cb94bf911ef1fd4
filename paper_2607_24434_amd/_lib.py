"""ctypes binding of libdraftexpert.so: argument marshalling only.

Every function below has the name of the C entry point it calls, takes torch
tensors (device memory) or None for optional pointers, passes their
``data_ptr()`` and the current HIP stream, and raises ``DEError`` on a
non-zero return code.  There is no fallback: if the library is missing the
import of this module fails.
"""
from __future__ import annotations

import ctypes
import os

# torch first: its HIP runtime (SONAME libamdhip64.so.7) must be the one the
# dynamic linker resolves for this library too, so that one runtime owns the
# device memory and streams torch hands over.
import torch  # noqa: F401

HERE = os.path.dirname(os.path.abspath(__file__))
# DE_LIBRARY may name another build of the same ABI, e.g. the host-only
# sanitizer build of the expert cache, which exports a subset of the entry
# points (only those are bound then).
DEFAULT_LIB_PATH = os.path.join(HERE, "libdraftexpert.so")
LIB_PATH = os.environ.get("DE_LIBRARY") or DEFAULT_LIB_PATH

DE_SOFTMAX = 0
DE_SIGMOID = 1
DE_F32 = 0
DE_BF16 = 1
DE_Q4_0 = 2


def expert_bytes(wdtype: int, inter: int, hidden: int) -> int:
    """Bytes of one [G|U|D] expert block in the given weight format."""
    if wdtype == DE_Q4_0:
        return 3 * inter * hidden * 9 // 16
    return 3 * inter * hidden * (2 if wdtype == DE_BF16 else 4)

C_FUNCS = [
    "de_abi_version", "de_error_string", "de_hip_error_detail", "de_check_desc", "de_workspace_bytes",
    "de_workspace_init", "de_route_topk",
    "de_expert_union", "de_grouped_swiglu", "de_draft_layer", "de_verify_layer", "de_accept_workspace_bytes", "de_accept_len",
    "de_lm_head", "de_rmsnorm", "de_embed_gather", "de_dense_workspace_bytes", "de_dense_swiglu",
    "de_stream_probe", "de_time_next_phase",
    "de_check_model", "de_model_workspace_bytes", "de_model_forward", "de_spec_step",
    "de_greedy_decode", "de_cache_create", "de_cache_destroy", "de_cache_reset",
    "de_cache_begin_block", "de_cache_prefetch", "de_cache_ensure", "de_cache_release",
    "de_cache_table", "de_cache_stats", "de_cache_slots", "de_spec_step_cached",
    "de_confidence", "de_expansion", "de_spec_step_trunc", "de_draft_layer_topr",
    "de_residual_target", "de_layer_router_logits", "de_row_kl", "de_distill_signals",
    "de_layer_status", "de_model_status", "de_noalloc_scratch_bytes", "de_verify_layer_noalloc",
    "de_verify_single_launch",
]
DE_PHASE_GATEUP = 0
DE_PHASE_DOWN = 1
DE_PHASE_LAYER = 2
DE_PHASE_DRAFT_PASS = 3
DE_TARGET = 0
DE_DRAFT = 1
DE_NEED_DRAFT = 0
DE_NEED_VERIFY = 1
DE_BUDGET_CACHE = -1


class DEError(RuntimeError):
    def __init__(self, fn: str, code: int, msg: str):
        super().__init__(f"{fn} failed with {code}: {msg}")
        self.code = code


class MoEDesc(ctypes.Structure):
    _fields_ = [
        ("hidden", ctypes.c_int32), ("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32),
        ("inter", ctypes.c_int32), ("shared_inter", ctypes.c_int32),
        ("draft_inter", ctypes.c_int32), ("score_func", ctypes.c_int32),
        ("norm_topk", ctypes.c_int32), ("routed_scale", ctypes.c_float),
        ("wdtype", ctypes.c_int32),
    ]


class ExpertTable(ctypes.Structure):
    _fields_ = [
        ("base", ctypes.c_void_p), ("slot_stride_bytes", ctypes.c_int64),
        ("slot_of_expert", ctypes.c_void_p), ("n_slots", ctypes.c_int32),
    ]


class Epilogue(ctypes.Structure):
    _fields_ = [("residual", ctypes.c_void_p), ("normed", ctypes.c_void_p), ("eps", ctypes.c_float)]


class LayerWeights(ctypes.Structure):
    _fields_ = [
        ("w_router", ctypes.c_void_p), ("bias", ctypes.c_void_p), ("routed", ExpertTable),
        ("shared_w", ctypes.c_void_p), ("draft_w", ctypes.c_void_p), ("gamma", ctypes.c_float),
    ]


class Model(ctypes.Structure):
    _fields_ = [
        ("moe", MoEDesc), ("n_layers", ctypes.c_int32), ("vocab", ctypes.c_int32),
        ("dense_inter", ctypes.c_int32), ("dense_wdtype", ctypes.c_int32), ("eps", ctypes.c_float),
        ("emb", ctypes.c_void_p), ("dense_w", ctypes.c_void_p), ("lm_head", ctypes.c_void_p),
        ("layers", ctypes.POINTER(LayerWeights)), ("draft_topr", ctypes.c_int32),
    ]


class CacheCfg(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("n_experts", ctypes.c_int32), ("n_slots", ctypes.c_int32),
        ("fake_copies", ctypes.c_int32), ("expert_bytes", ctypes.c_int64),
        ("slot_stride_bytes", ctypes.c_int64), ("host_pool", ctypes.c_void_p),
        ("slot_pool", ctypes.c_void_p), ("slot_map", ctypes.c_void_p),
    ]


CACHE_COUNTS = ("prefetch_issued", "prefetch_used", "prefetch_wasted", "prefetch_skipped",
                "draft_needed", "draft_hits", "verify_needed", "verify_hits", "demand_loads",
                "evictions", "bytes_copied")


class TruncCfg(ctypes.Structure):
    _fields_ = [("tau", ctypes.c_float), ("budget", ctypes.c_int32), ("slots", ctypes.c_int32),
                ("prefetch", ctypes.c_int32)]


class CacheCounts(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in CACHE_COUNTS] + [
        ("stall_us", ctypes.c_double), ("draft_layers", ctypes.c_int64),
        ("draft_layer_us", ctypes.c_double), ("verify_layers", ctypes.c_int64),
        ("verify_layer_us", ctypes.c_double)]


def _load(path: str = LIB_PATH, strict: bool = True):
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python paper_2607_24434_amd/build.py`")
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    I = ctypes.c_int
    F = ctypes.c_float
    SZ = ctypes.c_size_t
    DP = ctypes.POINTER(MoEDesc)
    TP = ctypes.POINTER(ExpertTable)
    EP = ctypes.POINTER(Epilogue)
    MP = ctypes.POINTER(Model)
    CP = ctypes.POINTER(CacheCfg)
    KP = ctypes.POINTER(CacheCounts)
    I32P = ctypes.POINTER(ctypes.c_int32)
    sig = {
        "de_abi_version": (I, []),
        "de_error_string": (ctypes.c_char_p, [I]),
        "de_hip_error_detail": (ctypes.c_char_p, []),
        "de_check_desc": (I, [DP]),
        "de_workspace_bytes": (SZ, [DP, I]),
        "de_workspace_init": (I, [P, SZ, P]),
        "de_route_topk": (I, [DP, I, P, P, P, P, P, P, SZ, P]),
        "de_expert_union": (I, [I, I, I, P, P, P, P, P, P, P, P, P]),
        "de_grouped_swiglu": (I, [DP, I, P, TP, P, P, P, P, P, P, P, P, EP, P, SZ, P]),
        "de_draft_layer": (I, [DP, I, P, P, P, TP, P, P, F, P, P, P, EP, P, SZ, P]),
        "de_draft_layer_topr": (I, [DP, I, P, P, P, TP, P, P, F, I, P, P, P, EP, P, SZ, P]),
        "de_residual_target": (I, [DP, I, P, SZ, P, P]),
        "de_layer_router_logits": (I, [DP, I, P, SZ, P, P]),
        "de_row_kl": (I, [I, I, P, I, P, I, P, I, F, P, P, P]),
        "de_distill_signals": (I, [MP, I, P, F, P, P, P, P, P, SZ, P]),
        "de_verify_layer": (I, [DP, I, P, P, P, TP, P, P, P, P, P, P, P, P, P, P, EP, P, SZ, P]),
        "de_accept_workspace_bytes": (SZ, [I, I]),
        "de_accept_len": (I, [I, I, P, P, P, P, P, SZ, P]),
        "de_lm_head": (I, [I, I, I, P, P, P, P]),
        "de_rmsnorm": (I, [I, I, P, F, P, P]),
        "de_embed_gather": (I, [I, I, I, P, P, P, P, F, P, P]),
        "de_layer_status": (I, [P, SZ, P]),
        "de_noalloc_scratch_bytes": (SZ, []),
        "de_verify_layer_noalloc": (I, [DP, I, P, P, P, TP, P, P, P, P, P, P, P, P, P, P, EP, P]),
        "de_model_status": (I, [MP, P, SZ, P]),
        "de_dense_workspace_bytes": (SZ, [I, I, I]),
        "de_dense_swiglu": (I, [I, I, I, I, P, P, P, EP, P, SZ, P]),
        "de_stream_probe": (I, [P, SZ, P, P]),
        "de_time_next_phase": (I, [I, P, P]),
        "de_verify_single_launch": (I, [DP, I]),
        "de_check_model": (I, [MP]),
        "de_model_workspace_bytes": (SZ, [MP, I]),
        "de_model_forward": (I, [MP, I, P, I, P, P, P, P, SZ, P]),
        "de_spec_step": (I, [MP, I, P, P, P, P, P, P, SZ, P]),
        "de_greedy_decode": (I, [MP, I, P, P, SZ, P]),
        "de_cache_create": (I, [CP, ctypes.POINTER(P)]),
        "de_cache_destroy": (I, [P]),
        "de_cache_reset": (I, [P]),
        "de_cache_begin_block": (I, [P]),
        "de_cache_prefetch": (I, [P, I, I32P, I]),
        "de_cache_ensure": (I, [P, I, I32P, I, I, P]),
        "de_cache_release": (I, [P, I, P]),
        "de_cache_table": (I, [P, I, TP]),
        "de_cache_stats": (I, [P, KP]),
        "de_cache_slots": (I, [P, I, I32P]),
        "de_spec_step_cached": (I, [MP, P, I, P, P, P, P, P, P, SZ, P]),
        "de_confidence": (I, [I, I, P, P, P]),
        "de_expansion": (I, [I, I, I, P, P, I, P, F, I, I, P, P]),
        "de_spec_step_trunc": (I, [MP, P, I, ctypes.POINTER(TruncCfg), P, P, P, I32P, P, P, P,
                                   P, P, SZ, P]),
    }
    for name, (res, args) in sig.items():
        if not strict and not hasattr(lib, name):
            continue
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


LIB = _load(LIB_PATH, strict=LIB_PATH == DEFAULT_LIB_PATH)


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    return torch.cuda.current_stream().cuda_stream


def _check(fn: str, rc: int):
    if rc != 0:
        msg = LIB.de_error_string(rc).decode()
        if rc == -3:
            msg += f" ({LIB.de_hip_error_detail().decode()})"
        raise DEError(fn, rc, msg)


def make_desc(hidden, n_experts, top_k, inter, shared_inter, draft_inter, score_func, norm_topk,
              routed_scale=1.0, wdtype=DE_BF16) -> MoEDesc:
    return MoEDesc(int(hidden), int(n_experts), int(top_k), int(inter), int(shared_inter),
                   int(draft_inter), int(score_func), int(bool(norm_topk)), float(routed_scale),
                   int(wdtype))


def make_table(base, slot_stride_bytes: int, slot_of_expert=None, n_slots: int = 0) -> ExpertTable:
    return ExpertTable(_ptr(base), int(slot_stride_bytes), _ptr(slot_of_expert), int(n_slots))


def make_epilogue(residual=None, normed=None, eps: float = 1e-6):
    if residual is None and normed is None:
        return None
    return Epilogue(_ptr(residual), _ptr(normed), float(eps))


def _epi_arg(epi):
    return None if epi is None else ctypes.byref(epi)


def de_abi_version() -> int:
    return LIB.de_abi_version()


def de_error_string(code: int) -> str:
    return LIB.de_error_string(code).decode()


def de_check_desc(desc: MoEDesc) -> int:
    return LIB.de_check_desc(ctypes.byref(desc))


def de_workspace_bytes(desc: MoEDesc, T: int) -> int:
    return LIB.de_workspace_bytes(ctypes.byref(desc), int(T))


def de_workspace_init(ws, stream=None):
    _check("de_workspace_init", LIB.de_workspace_init(_ptr(ws), ws.numel(), _stream(stream)))


def workspace(desc, T, device="cuda"):
    """A zero-initialised workspace tensor for layer calls of up to T positions."""
    ws = torch.empty(de_workspace_bytes(desc, T), dtype=torch.uint8, device=device)
    de_workspace_init(ws)
    return ws


def de_route_topk(desc, T, x, w_router, bias, topk_idx, topk_gate, ws, stream=None):
    _check("de_route_topk", LIB.de_route_topk(
        ctypes.byref(desc), int(T), _ptr(x), _ptr(w_router), _ptr(bias), _ptr(topk_idx),
        _ptr(topk_gate), _ptr(ws), ws.numel() if ws is not None else 0, _stream(stream)))


def de_expert_union(T, k, N, topk_idx, topk_gate, n_union, union_ids, offsets, tok_list,
                    gate_list, pair_pos, stream=None):
    _check("de_expert_union", LIB.de_expert_union(
        int(T), int(k), int(N), _ptr(topk_idx), _ptr(topk_gate), _ptr(n_union), _ptr(union_ids),
        _ptr(offsets), _ptr(tok_list), _ptr(gate_list), _ptr(pair_pos), _stream(stream)))


def de_grouped_swiglu(desc, T, x, table, n_union, union_ids, offsets, tok_list, gate_list,
                      pair_pos, shared_w, y, ws, epi=None, stream=None):
    _check("de_grouped_swiglu", LIB.de_grouped_swiglu(
        ctypes.byref(desc), int(T), _ptr(x), ctypes.byref(table), _ptr(n_union), _ptr(union_ids),
        _ptr(offsets), _ptr(tok_list), _ptr(gate_list), _ptr(pair_pos), _ptr(shared_w), _ptr(y),
        _epi_arg(epi), _ptr(ws), ws.numel(), _stream(stream)))


def de_draft_layer(desc, T, x, w_router, bias, table, shared_w, draft_w, gamma, y, pred_idx,
                   pred_gate, ws, epi=None, stream=None):
    _check("de_draft_layer", LIB.de_draft_layer(
        ctypes.byref(desc), int(T), _ptr(x), _ptr(w_router), _ptr(bias), ctypes.byref(table),
        _ptr(shared_w), _ptr(draft_w), float(gamma), _ptr(y), _ptr(pred_idx), _ptr(pred_gate),
        _epi_arg(epi), _ptr(ws), ws.numel(), _stream(stream)))


def de_draft_layer_topr(desc, T, x, w_router, bias, table, shared_w, draft_w, gamma, r, y,
                        pred_idx, pred_gate, ws, epi=None, stream=None):
    _check("de_draft_layer_topr", LIB.de_draft_layer_topr(
        ctypes.byref(desc), int(T), _ptr(x), _ptr(w_router), _ptr(bias), ctypes.byref(table),
        _ptr(shared_w), _ptr(draft_w), float(gamma), int(r), _ptr(y), _ptr(pred_idx),
        _ptr(pred_gate), _epi_arg(epi), _ptr(ws), ws.numel(), _stream(stream)))


def de_verify_layer(desc, T, x, w_router, bias, table, shared_w, y, topk_idx=None, topk_gate=None,
                    n_union=None, union_ids=None, offsets=None, tok_list=None, gate_list=None,
                    pair_pos=None, ws=None, epi=None, stream=None):
    _check("de_verify_layer", LIB.de_verify_layer(
        ctypes.byref(desc), int(T), _ptr(x), _ptr(w_router), _ptr(bias), ctypes.byref(table),
        _ptr(shared_w), _ptr(y), _ptr(topk_idx), _ptr(topk_gate), _ptr(n_union), _ptr(union_ids),
        _ptr(offsets), _ptr(tok_list), _ptr(gate_list), _ptr(pair_pos), _epi_arg(epi), _ptr(ws),
        ws.numel() if ws is not None else 0, _stream(stream)))


def de_noalloc_scratch_bytes() -> int:
    return LIB.de_noalloc_scratch_bytes()


def de_verify_layer_noalloc(desc, T, x, w_router, bias, table, shared_w, y, topk_idx=None,
                            topk_gate=None, n_union=None, union_ids=None, offsets=None,
                            tok_list=None, gate_list=None, pair_pos=None, epi=None, stream=None):
    _check("de_verify_layer_noalloc", LIB.de_verify_layer_noalloc(
        ctypes.byref(desc), int(T), _ptr(x), _ptr(w_router), _ptr(bias), ctypes.byref(table),
        _ptr(shared_w), _ptr(y), _ptr(topk_idx), _ptr(topk_gate), _ptr(n_union), _ptr(union_ids),
        _ptr(offsets), _ptr(tok_list), _ptr(gate_list), _ptr(pair_pos), _epi_arg(epi),
        _stream(stream)))


def de_accept_workspace_bytes(K, V) -> int:
    return LIB.de_accept_workspace_bytes(int(K), int(V))


def accept_workspace(K, V, device="cuda"):
    """A zero-initialised scratch tensor for de_accept_len with up to K drafts."""
    ws = torch.empty(de_accept_workspace_bytes(K, V), dtype=torch.uint8, device=device)
    de_workspace_init(ws)
    return ws


def de_accept_len(K, V, target_logits, draft_tokens, target_argmax, out, ws, stream=None):
    _check("de_accept_len", LIB.de_accept_len(
        int(K), int(V), _ptr(target_logits), _ptr(draft_tokens), _ptr(target_argmax), _ptr(out),
        _ptr(ws), ws.numel(), _stream(stream)))


def de_lm_head(T, H, V, x, w_lm, logits, stream=None):
    _check("de_lm_head", LIB.de_lm_head(int(T), int(H), int(V), _ptr(x), _ptr(w_lm), _ptr(logits),
                                        _stream(stream)))


def de_rmsnorm(T, H, x, eps, out, stream=None):
    _check("de_rmsnorm", LIB.de_rmsnorm(int(T), int(H), _ptr(x), float(eps), _ptr(out),
                                        _stream(stream)))


def de_embed_gather(T, H, V, tokens, emb, h, normed=None, eps=1e-6, status=None, stream=None):
    _check("de_embed_gather", LIB.de_embed_gather(int(T), int(H), int(V), _ptr(tokens), _ptr(emb),
                                                  _ptr(h), _ptr(normed), float(eps),
                                                  _ptr(status), _stream(stream)))


def de_layer_status(ws, stream=None) -> int:
    """The workspace's device status as a return code (0, or -5 / -1); waits and clears."""
    return LIB.de_layer_status(_ptr(ws), ws.numel(), _stream(stream))


def de_model_status(model, ws, stream=None) -> int:
    return LIB.de_model_status(ctypes.byref(model), _ptr(ws), ws.numel(), _stream(stream))


def de_dense_workspace_bytes(T, H, I) -> int:
    return LIB.de_dense_workspace_bytes(int(T), int(H), int(I))


def de_dense_swiglu(T, H, I, wdtype, x, w, y, ws, epi=None, stream=None):
    _check("de_dense_swiglu", LIB.de_dense_swiglu(
        int(T), int(H), int(I), int(wdtype), _ptr(x), _ptr(w), _ptr(y), _epi_arg(epi), _ptr(ws),
        ws.numel(), _stream(stream)))


def de_stream_probe(buf, nbytes, sink, stream=None):
    _check("de_stream_probe", LIB.de_stream_probe(_ptr(buf), int(nbytes), _ptr(sink),
                                                  _stream(stream)))


def de_time_next_phase(phase, start_event, stop_event):
    """Arm the one-shot phase timer with torch.cuda.Event objects (already recorded once)."""
    _check("de_time_next_phase", LIB.de_time_next_phase(
        int(phase), None if start_event is None else start_event.cuda_event,
        None if stop_event is None else stop_event.cuda_event))


def de_verify_single_launch(desc, T):
    """True when the verify layer of this shape runs as one launch."""
    return bool(LIB.de_verify_single_launch(ctypes.byref(desc), int(T)))


def make_model(desc, layers, vocab, emb, lm_head, dense_w=None, dense_inter=0,
               dense_wdtype=DE_BF16, eps=1e-6, draft_topr=1):
    """A ``Model`` struct; ``layers`` is a list of dicts with the keys w_router,
    bias, table (an ExpertTable), shared_w, draft_w, gamma.  The returned
    struct keeps the layer array alive."""
    arr = (LayerWeights * max(1, len(layers)))()
    for i, l in enumerate(layers):
        arr[i] = LayerWeights(_ptr(l["w_router"]), _ptr(l.get("bias")), l["table"],
                              _ptr(l.get("shared_w")), _ptr(l.get("draft_w")),
                              float(l.get("gamma", 1.0)))
    m = Model(desc, len(layers), int(vocab), int(dense_inter), int(dense_wdtype), float(eps),
              _ptr(emb), _ptr(dense_w), _ptr(lm_head), arr, int(draft_topr))
    m._layers = arr
    return m


def de_check_model(model) -> int:
    return LIB.de_check_model(ctypes.byref(model))


def de_model_workspace_bytes(model, T) -> int:
    return LIB.de_model_workspace_bytes(ctypes.byref(model), int(T))


def model_workspace(model, T, device="cuda"):
    """A zero-initialised scratch tensor for the model calls with up to T positions."""
    n = de_model_workspace_bytes(model, T)
    if n == 0:
        _check("de_model_workspace_bytes", de_check_model(model) or -1)
    ws = torch.empty(n, dtype=torch.uint8, device=device)
    de_workspace_init(ws)
    return ws


def de_model_forward(model, T, tokens, mode, logits, argmax=None, n_union=None, ws=None,
                     stream=None):
    _check("de_model_forward", LIB.de_model_forward(
        ctypes.byref(model), int(T), _ptr(tokens), int(mode), _ptr(logits), _ptr(argmax),
        _ptr(n_union), _ptr(ws), ws.numel() if ws is not None else 0, _stream(stream)))


def de_spec_step(model, K, block, target_argmax, out, n_union=None, pred_idx=None, ws=None,
                 stream=None):
    _check("de_spec_step", LIB.de_spec_step(
        ctypes.byref(model), int(K), _ptr(block), _ptr(target_argmax), _ptr(out), _ptr(n_union),
        _ptr(pred_idx), _ptr(ws), ws.numel() if ws is not None else 0, _stream(stream)))


def de_greedy_decode(model, n_steps, tokens, ws=None, stream=None):
    _check("de_greedy_decode", LIB.de_greedy_decode(
        ctypes.byref(model), int(n_steps), _ptr(tokens), _ptr(ws),
        ws.numel() if ws is not None else 0, _stream(stream)))


def _i32(values):
    vals = [int(v) for v in values]
    return (ctypes.c_int32 * max(1, len(vals)))(*vals), len(vals)


class ExpertCache:
    """Owner of a ``de_cache``: per-layer HBM slots over a host pool of expert blocks.

    ``host_pool`` is a pinned CPU tensor [L, N, expert_bytes] (uint8 view of the
    blocks).  With ``fake=True`` the slot pool and slot map are CPU tensors and
    copies are host memcpy (bookkeeping without a GPU)."""

    def __init__(self, n_layers, n_experts, n_slots, expert_bytes, host_pool, fake=False,
                 device="cuda"):
        stride = (int(expert_bytes) + 255) // 256 * 256
        dev = "cpu" if fake else device
        self.slot_pool = torch.empty(n_layers * n_slots * stride, dtype=torch.uint8, device=dev)
        self.slot_map = torch.empty(n_layers * n_experts, dtype=torch.int32, device=dev)
        self.host_pool = host_pool
        self.cfg = CacheCfg(int(n_layers), int(n_experts), int(n_slots), int(bool(fake)),
                            int(expert_bytes), stride, _ptr(host_pool), _ptr(self.slot_pool),
                            _ptr(self.slot_map))
        self.n_layers, self.n_experts, self.n_slots = int(n_layers), int(n_experts), int(n_slots)
        self.stride = stride
        h = ctypes.c_void_p()
        _check("de_cache_create", LIB.de_cache_create(ctypes.byref(self.cfg), ctypes.byref(h)))
        self.handle = h

    def close(self):
        if self.handle is not None and self.handle.value:
            _check("de_cache_destroy", LIB.de_cache_destroy(self.handle))
        self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:  # noqa: BLE001
            pass

    def reset(self):
        _check("de_cache_reset", LIB.de_cache_reset(self.handle))

    def begin_block(self):
        _check("de_cache_begin_block", LIB.de_cache_begin_block(self.handle))

    def prefetch(self, layer, experts):
        arr, n = _i32(experts)
        _check("de_cache_prefetch", LIB.de_cache_prefetch(self.handle, int(layer), arr, n))

    def ensure(self, layer, needed, purpose, stream=None):
        arr, n = _i32(needed)
        s = None if self.cfg.fake_copies else _stream(stream)
        _check("de_cache_ensure", LIB.de_cache_ensure(self.handle, int(layer), arr, n,
                                                      int(purpose), s))

    def release(self, layer, stream=None):
        s = None if self.cfg.fake_copies else _stream(stream)
        _check("de_cache_release", LIB.de_cache_release(self.handle, int(layer), s))

    def table(self, layer) -> ExpertTable:
        t = ExpertTable()
        _check("de_cache_table", LIB.de_cache_table(self.handle, int(layer), ctypes.byref(t)))
        return t

    def stats(self) -> dict:
        k = CacheCounts()
        _check("de_cache_stats", LIB.de_cache_stats(self.handle, ctypes.byref(k)))
        return {n: getattr(k, n) for n, _ in CacheCounts._fields_}

    def slots(self, layer) -> list:
        arr = (ctypes.c_int32 * self.n_experts)()
        _check("de_cache_slots", LIB.de_cache_slots(self.handle, int(layer), arr))
        return list(arr)


def de_spec_step_cached(model, cache, K, block, target_argmax, out, n_union=None, pred_idx=None,
                        ws=None, stream=None):
    _check("de_spec_step_cached", LIB.de_spec_step_cached(
        ctypes.byref(model), cache.handle, int(K), _ptr(block), _ptr(target_argmax), _ptr(out),
        _ptr(n_union), _ptr(pred_idx), _ptr(ws), ws.numel() if ws is not None else 0,
        _stream(stream)))


def de_confidence(T, V, logits, q, stream=None):
    _check("de_confidence", LIB.de_confidence(int(T), int(V), _ptr(logits), _ptr(q),
                                              _stream(stream)))


def de_expansion(L, k, N, pred_idx, uhat, first, q, tau, budget, slots, out, stream=None):
    _check("de_expansion", LIB.de_expansion(
        int(L), int(k), int(N), _ptr(pred_idx), _ptr(uhat), int(bool(first)), _ptr(q),
        float(tau), int(budget), int(slots), _ptr(out), _stream(stream)))


def de_spec_step_trunc(model, cache, k_max, tau, budget, slots, block, target_argmax, out,
                       pred_idx, q, n_union=None, trace=None, ws=None, stream=None,
                       prefetch=True) -> int:
    """Returns the number of kept drafts."""
    cfg = TruncCfg(float(tau), int(budget), int(slots), int(bool(prefetch)))
    nd = ctypes.c_int32(0)
    _check("de_spec_step_trunc", LIB.de_spec_step_trunc(
        ctypes.byref(model), cache.handle if cache is not None else None, int(k_max),
        ctypes.byref(cfg), _ptr(block), _ptr(target_argmax), _ptr(out), ctypes.byref(nd),
        _ptr(n_union), _ptr(pred_idx), _ptr(q), _ptr(trace), _ptr(ws),
        ws.numel() if ws is not None else 0, _stream(stream)))
    return int(nd.value)


def de_residual_target(desc, T, ws, m_star, stream=None):
    _check("de_residual_target", LIB.de_residual_target(
        ctypes.byref(desc), int(T), _ptr(ws), ws.numel(), _ptr(m_star), _stream(stream)))


def de_layer_router_logits(desc, T, ws, z, stream=None):
    _check("de_layer_router_logits", LIB.de_layer_router_logits(
        ctypes.byref(desc), int(T), _ptr(ws), ws.numel(), _ptr(z), _stream(stream)))


def de_row_kl(rows, n, a, lda, b, ldb, bias, sigmoid, tau, kl, ce=None, stream=None):
    _check("de_row_kl", LIB.de_row_kl(int(rows), int(n), _ptr(a), int(lda), _ptr(b), int(ldb),
                                      _ptr(bias), int(bool(sigmoid)), float(tau), _ptr(kl),
                                      _ptr(ce), _stream(stream)))


def de_distill_signals(model, T, tokens, tau, m_star, router_kl, logit_kl, token_ce, ws=None,
                       stream=None):
    _check("de_distill_signals", LIB.de_distill_signals(
        ctypes.byref(model), int(T), _ptr(tokens), float(tau), _ptr(m_star), _ptr(router_kl),
        _ptr(logit_kl), _ptr(token_ce), _ptr(ws), ws.numel() if ws is not None else 0,
        _stream(stream)))
