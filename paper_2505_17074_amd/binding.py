"""ctypes binding of libspecverify.so: the C ABI under the same names.

Argument marshalling only -- every step of the verify path runs in the HIP
kernels of the library.  Loading fails loudly when the library is missing;
there is no fallback implementation.
"""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libspecverify.so")

SPEC_OK, SPEC_ERR_INVALID_ARG, SPEC_ERR_UNSUPPORTED, SPEC_ERR_WORKSPACE, SPEC_ERR_HIP = range(5)
SPEC_F32, SPEC_BF16 = 0, 1
SPEC_TREE_INDEPENDENT, SPEC_TREE_SEQUENTIAL = 0, 1
SPEC_MAX_DRAFT = 16
SPEC_MAX_TREE_NODES = 32
SPEC_NOALLOC_SCRATCH_BYTES = 32 << 20
SPEC_NOALLOC_STAGING_BYTES = 1 << 20

EXPORTS = ("spec_workspace_bytes", "spec_verify_attn", "spec_accept", "spec_verify",
           "spec_status_str", "spec_abi_version", "spec_stream_read_probe", "spec_accept_floor_probe",
           "spec_accept_floor_probe_bytes", "spec_verify_noalloc",
           "spec_lm_head_accept", "spec_lm_head_workspace_bytes",
           "spec_sched_create", "spec_sched_destroy", "spec_sched_submit", "spec_sched_next",
           "spec_sched_report", "spec_sched_query", "spec_sched_simulate")

SPEC_SCHED_FCFS, SPEC_SCHED_LP_SJF, SPEC_SCHED_SJF_EXACT, SPEC_SCHED_LAS, SPEC_SCHED_LAPS_SD = range(5)
SCHED_POLICY = {"fcfs": SPEC_SCHED_FCFS, "lp_sjf": SPEC_SCHED_LP_SJF, "sjf_exact": SPEC_SCHED_SJF_EXACT,
                "las": SPEC_SCHED_LAS, "laps_sd": SPEC_SCHED_LAPS_SD}


class SpecRequests(C.Structure):
    _fields_ = [("num_requests", C.c_int32),
                ("ctx_len", C.POINTER(C.c_int32)),
                ("draft_len", C.POINTER(C.c_int32)),
                ("tree_nodes", C.c_int32),
                ("tree_parent", C.POINTER(C.c_int32)),
                ("node_count", C.POINTER(C.c_int32)),
                ("tree_parents", C.POINTER(C.c_int32))]


class SpecAttnArgs(C.Structure):
    _fields_ = [("num_q_heads", C.c_int32),
                ("num_kv_heads", C.c_int32),
                ("head_dim", C.c_int32),
                ("dtype", C.c_int),
                ("scale", C.c_float),
                ("q", C.c_void_p),
                ("q_stride_tok", C.c_int64),
                ("q_stride_head", C.c_int64),
                ("k", C.c_void_p),
                ("v", C.c_void_p),
                ("kv_stride_tok", C.c_int64),
                ("kv_stride_head", C.c_int64),
                ("out", C.c_void_p),
                ("split_kv", C.c_int32),
                ("event_begin", C.c_void_p),
                ("event_end", C.c_void_p),
                ("block_table", C.c_void_p),
                ("block_stride", C.c_int32),
                ("page_tokens", C.c_int32),
                ("num_pages", C.c_int32),
                ("pad0", C.c_int32)]


class SpecAcceptArgs(C.Structure):
    _fields_ = [("vocab", C.c_int32),
                ("dtype", C.c_int),
                ("target_logits", C.c_void_p),
                ("logits_stride", C.c_int64),
                ("draft_probs", C.c_void_p),
                ("probs_stride", C.c_int64),
                ("draft_tokens", C.c_void_p),
                ("uniforms", C.c_void_p),
                ("accepted_len", C.c_void_p),
                ("next_token", C.c_void_p),
                ("accepted_node", C.c_void_p),
                ("event_begin", C.c_void_p),
                ("event_end", C.c_void_p),
                ("event_mid", C.c_void_p),
                ("tree_rule", C.c_int32),
                ("pad0", C.c_int32)]


class SpecLmHeadArgs(C.Structure):
    _fields_ = [("hidden_dim", C.c_int32),
                ("pad0", C.c_int32),
                ("hidden", C.c_void_p),
                ("hidden_stride", C.c_int64),
                ("weight", C.c_void_p),
                ("weight_stride", C.c_int64),
                ("event_begin", C.c_void_p),
                ("event_end", C.c_void_p)]


class SpecSchedParams(C.Structure):
    _fields_ = [("K", C.c_int32),
                ("M", C.c_int32),
                ("S1_up_us", C.c_int64),
                ("gamma", C.c_int32),
                ("pad0", C.c_int32),
                ("delta", C.c_double),
                ("t_ssm_us", C.c_int64),
                ("t_llm_us", C.c_int64),
                ("swap_us_per_token", C.c_int64)]


class SpecSchedState(C.Structure):
    _fields_ = [("attained_us", C.c_int64),
                ("queue", C.c_int32),
                ("perceptible", C.c_int32),
                ("finished", C.c_int32),
                ("rounds", C.c_int32),
                ("A", C.c_double),
                ("T_est_us", C.c_double)]


class SpecSchedRequest(C.Structure):
    _fields_ = [("arrival_us", C.c_int64),
                ("round_us", C.c_int64),
                ("prompt_tokens", C.c_int32),
                ("out_len", C.c_int32),
                ("pred_len", C.c_int32),
                ("draft", C.c_int32),
                ("accepted", C.POINTER(C.c_int32)),
                ("n_accepted", C.c_int32),
                ("pad0", C.c_int32)]


class SpecSchedResult(C.Structure):
    _fields_ = [("completion_us", C.POINTER(C.c_int64)),
                ("round_req", C.POINTER(C.c_int32)),
                ("round_start_us", C.POINTER(C.c_int64)),
                ("max_rounds", C.c_int64),
                ("n_rounds", C.c_int64),
                ("switches", C.c_int64),
                ("switch_us", C.c_int64),
                ("perceptible", C.POINTER(C.c_int32)),
                ("A", C.POINTER(C.c_double)),
                ("T_est_us", C.POINTER(C.c_double))]


class SpecError(RuntimeError):
    def __init__(self, status: int, where: str, text: str):
        super().__init__(f"{where}: {text} (status {status})")
        self.status = status


_lib = None


def load(path: str = LIB_PATH) -> C.CDLL:
    """Load the built library (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with paper_2505_17074_amd/build.py "
                           "(or __graft_entry__.build()); there is no fallback path")
    lib = C.CDLL(path)
    P = C.POINTER
    lib.spec_workspace_bytes.argtypes = [P(SpecRequests), P(SpecAttnArgs), P(SpecAcceptArgs),
                                         P(C.c_size_t), P(C.c_size_t)]
    lib.spec_workspace_bytes.restype = C.c_int
    lib.spec_verify_attn.argtypes = [P(SpecRequests), P(SpecAttnArgs), C.c_void_p, C.c_size_t,
                                     C.c_void_p, C.c_size_t, C.c_void_p]
    lib.spec_verify_attn.restype = C.c_int
    lib.spec_accept.argtypes = [P(SpecRequests), P(SpecAcceptArgs), C.c_void_p, C.c_size_t,
                                C.c_void_p, C.c_size_t, C.c_void_p]
    lib.spec_accept.restype = C.c_int
    lib.spec_verify.argtypes = [P(SpecRequests), P(SpecAttnArgs), P(SpecAcceptArgs), C.c_void_p, C.c_size_t,
                                C.c_void_p, C.c_size_t, C.c_void_p]
    lib.spec_verify.restype = C.c_int
    lib.spec_verify_noalloc.argtypes = [P(SpecRequests), P(SpecAttnArgs), P(SpecAcceptArgs), C.c_void_p]
    lib.spec_verify_noalloc.restype = C.c_int
    lib.spec_lm_head_accept.argtypes = [P(SpecRequests), P(SpecLmHeadArgs), P(SpecAcceptArgs), C.c_void_p,
                                        C.c_size_t, C.c_void_p, C.c_size_t, C.c_void_p]
    lib.spec_lm_head_accept.restype = C.c_int
    lib.spec_lm_head_workspace_bytes.argtypes = [P(SpecRequests), P(SpecLmHeadArgs), P(SpecAcceptArgs),
                                                 P(C.c_size_t), P(C.c_size_t)]
    lib.spec_lm_head_workspace_bytes.restype = C.c_int
    lib.spec_status_str.argtypes = [C.c_int]
    lib.spec_status_str.restype = C.c_char_p
    lib.spec_abi_version.argtypes = []
    lib.spec_abi_version.restype = C.c_int32
    lib.spec_stream_read_probe.argtypes = [C.c_void_p, C.c_size_t, C.c_void_p, C.c_int32, C.c_void_p]
    lib.spec_stream_read_probe.restype = C.c_int
    lib.spec_accept_floor_probe_bytes.argtypes = [C.c_int32, C.c_int32, C.c_int32]
    lib.spec_accept_floor_probe_bytes.restype = C.c_size_t
    lib.spec_accept_floor_probe.argtypes = [C.c_void_p, C.c_int64, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                            C.c_void_p, C.c_size_t, C.c_void_p, C.c_void_p]
    lib.spec_accept_floor_probe.restype = C.c_int
    lib.spec_sched_create.argtypes = [C.c_int32, P(SpecSchedParams), C.c_int32, P(C.c_void_p)]
    lib.spec_sched_create.restype = C.c_int
    lib.spec_sched_destroy.argtypes = [C.c_void_p]
    lib.spec_sched_destroy.restype = None
    lib.spec_sched_submit.argtypes = [C.c_void_p, C.c_int64, C.c_int32, C.c_int32, C.c_int32, C.c_int64,
                                      P(C.c_int32)]
    lib.spec_sched_submit.restype = C.c_int
    lib.spec_sched_next.argtypes = [C.c_void_p, C.c_int64, P(C.c_int32)]
    lib.spec_sched_next.restype = C.c_int
    lib.spec_sched_report.argtypes = [C.c_void_p, C.c_int32, C.c_int32, C.c_int64, C.c_int32]
    lib.spec_sched_report.restype = C.c_int
    lib.spec_sched_query.argtypes = [C.c_void_p, C.c_int32, P(SpecSchedState)]
    lib.spec_sched_query.restype = C.c_int
    lib.spec_sched_simulate.argtypes = [P(SpecSchedRequest), C.c_int32, C.c_int32, P(SpecSchedParams),
                                        P(SpecSchedResult)]
    lib.spec_sched_simulate.restype = C.c_int
    _lib = lib
    return lib


def status_str(status: int) -> str:
    return load().spec_status_str(status).decode()


def check(status: int, where: str) -> None:
    if status != SPEC_OK:
        raise SpecError(status, where, status_str(status))


def _ref(x):
    return None if x is None else C.byref(x)


def spec_workspace_bytes(req: SpecRequests, attn: SpecAttnArgs | None, acc: SpecAcceptArgs | None):
    """Returns (status, device_bytes, host_bytes)."""
    dev, host = C.c_size_t(0), C.c_size_t(0)
    st = load().spec_workspace_bytes(C.byref(req), _ref(attn), _ref(acc), C.byref(dev), C.byref(host))
    return st, dev.value, host.value


def spec_verify_attn(req, attn, ws: int, ws_bytes: int, staging: int, staging_bytes: int, stream: int) -> int:
    return load().spec_verify_attn(C.byref(req), _ref(attn), ws, ws_bytes, staging, staging_bytes, stream)


def spec_accept(req, acc, ws: int, ws_bytes: int, staging: int, staging_bytes: int, stream: int) -> int:
    return load().spec_accept(C.byref(req), _ref(acc), ws, ws_bytes, staging, staging_bytes, stream)


def spec_verify(req, attn, acc, ws: int, ws_bytes: int, staging: int, staging_bytes: int, stream: int) -> int:
    return load().spec_verify(C.byref(req), _ref(attn), _ref(acc), ws, ws_bytes, staging, staging_bytes, stream)


def spec_verify_noalloc(req, attn, acc, stream: int) -> int:
    return load().spec_verify_noalloc(C.byref(req), _ref(attn), _ref(acc), stream)


def spec_lm_head_workspace_bytes(req: SpecRequests, lm: SpecLmHeadArgs, acc: SpecAcceptArgs):
    """Returns (status, device_bytes, host_bytes)."""
    dev, host = C.c_size_t(0), C.c_size_t(0)
    st = load().spec_lm_head_workspace_bytes(C.byref(req), _ref(lm), _ref(acc), C.byref(dev), C.byref(host))
    return st, dev.value, host.value


def spec_lm_head_accept(req, lm, acc, ws: int, ws_bytes: int, staging: int, staging_bytes: int, stream: int) -> int:
    return load().spec_lm_head_accept(C.byref(req), _ref(lm), _ref(acc), ws, ws_bytes, staging, staging_bytes, stream)


def spec_abi_version() -> int:
    return int(load().spec_abi_version())


def spec_stream_read_probe(src, nbytes, out, blocks, stream):
    return load().spec_stream_read_probe(src, nbytes, out, blocks, stream)


def spec_accept_floor_probe_bytes(V, num_rows, B):
    return int(load().spec_accept_floor_probe_bytes(V, num_rows, B))


def spec_accept_floor_probe(rows, row_stride, elem_bytes, V, num_rows, B, ws, ws_bytes, out, stream):
    return load().spec_accept_floor_probe(rows, row_stride, elem_bytes, V, num_rows, B, ws, ws_bytes, out, stream)


def make_requests(ctx_len, draft_len=None, tree_parent=None, tree_parents=None):
    """SpecRequests over host int32 arrays; the arrays are kept alive on the struct.
    Chains (draft_len), one shared tree (tree_parent) or a tree per request
    (tree_parents: one BFS parent array per request)."""
    import numpy as np
    ctx = np.ascontiguousarray(ctx_len, dtype=np.int32)
    r = SpecRequests()
    r.num_requests = int(ctx.shape[0])
    r.ctx_len = ctx.ctypes.data_as(C.POINTER(C.c_int32))
    keep = [ctx]
    if draft_len is not None:
        k = np.ascontiguousarray(draft_len, dtype=np.int32)
        r.draft_len = k.ctypes.data_as(C.POINTER(C.c_int32))
        keep.append(k)
    if tree_parent is not None:
        par = np.ascontiguousarray(tree_parent, dtype=np.int32)
        r.tree_nodes = int(par.shape[0])
        r.tree_parent = par.ctypes.data_as(C.POINTER(C.c_int32))
        keep.append(par)
    else:
        r.tree_nodes = 0
    if tree_parents is not None:
        cnt = np.ascontiguousarray([len(x) for x in tree_parents], dtype=np.int32)
        cat = np.ascontiguousarray(np.concatenate([np.asarray(x, np.int32) for x in tree_parents]), dtype=np.int32)
        r.node_count = cnt.ctypes.data_as(C.POINTER(C.c_int32))
        r.tree_parents = cat.ctypes.data_as(C.POINTER(C.c_int32))
        keep += [cnt, cat]
    r._keep = keep
    return r
