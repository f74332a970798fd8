"""The C ABI on a GPU-less host: exported symbols, status strings, and every
argument check (which must run before the first HIP call)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2505_17074_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "specverify.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        from paper_2505_17074_amd import build
        build.build()
    return B.load()


def _declared():
    names = []
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if h.endswith(".h"):
            text = open(os.path.join(ROOT, "include", h)).read()
            names += re.findall(r"SPEC_API\s+[\w\s\*]+?\b(spec_\w+)\s*\(", text)
    return names


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert set(names) == set(B.EXPORTS)
    for name in names:
        assert hasattr(lib, name), name
    nm = os.popen(f"nm -D --defined-only {B.LIB_PATH}").read()
    exported = set(re.findall(r"\bT (spec_\w+)", nm))
    assert exported == set(names)


def test_version_and_status_strings(lib):
    text = open(HEADER).read()
    assert B.spec_abi_version() == int(re.search(r"#define SPEC_ABI_VERSION (\d+)", text).group(1))
    assert B.status_str(B.SPEC_OK) == "ok"
    for st in range(1, 5):
        assert B.status_str(st) not in ("ok", "unknown status")
    assert B.status_str(99) == "unknown status"


FAKE = 1 << 20      # a 256-aligned fake device address; never dereferenced on these paths


def _attn(**kw):
    a = B.SpecAttnArgs()
    a.num_q_heads, a.num_kv_heads, a.head_dim, a.dtype = 8, 2, 128, B.SPEC_BF16
    a.q = a.k = a.v = a.out = FAKE
    a.q_stride_tok, a.q_stride_head = 8 * 128, 128
    a.kv_stride_tok, a.kv_stride_head = 2 * 128, 128
    for k, v in kw.items():
        setattr(a, k, v)
    return a


def _acc(**kw):
    a = B.SpecAcceptArgs()
    a.vocab, a.dtype = 1000, B.SPEC_F32
    a.target_logits = a.draft_probs = a.draft_tokens = a.uniforms = FAKE
    a.accepted_len = a.next_token = FAKE
    a.logits_stride = a.probs_stride = 1000
    for k, v in kw.items():
        setattr(a, k, v)
    return a


def _req(ctx=(5, 9), k=(2, 3), parent=None):
    return B.make_requests(np.array(ctx), None if parent is not None else np.array(k), parent)


def _ws(req, attn, acc):
    return B.spec_workspace_bytes(req, attn, acc)


def test_workspace_bytes_valid(lib):
    st, dev, host = _ws(_req(), _attn(), _acc())
    assert st == B.SPEC_OK and dev > 0 and host > 0 and dev % 256 == 0 and host <= dev
    # attention-only and acceptance-only need no more than the whole step
    st_a, dev_a, _ = _ws(_req(), _attn(), None)
    st_c, dev_c, _ = _ws(_req(), None, _acc())
    assert st_a == st_c == B.SPEC_OK and dev_a <= dev and dev_c <= dev
    # deterministic
    assert _ws(_req(), _attn(), _acc()) == (st, dev, host)
    # a forced split changes the partial area, not the verdict
    st2, dev2, _ = _ws(_req(ctx=(3000, 5000)), _attn(split_kv=256), None)
    st3, dev3, _ = _ws(_req(ctx=(3000, 5000)), _attn(split_kv=8192), None)
    assert st2 == st3 == B.SPEC_OK and dev2 > dev3


@pytest.mark.parametrize("req,expect", [
    (dict(ctx=(5, -1)), B.SPEC_ERR_INVALID_ARG),
    (dict(k=(2, 17)), B.SPEC_ERR_INVALID_ARG),
    (dict(k=(-1, 2)), B.SPEC_ERR_INVALID_ARG),
    (dict(k=(0, 16)), B.SPEC_OK),
    (dict(parent=[0, 0, 1]), B.SPEC_ERR_INVALID_ARG),
    (dict(parent=[-1, 0, 2]), B.SPEC_ERR_INVALID_ARG),
    (dict(parent=[-1, 0, 0, 1]), B.SPEC_OK),
    (dict(parent=[-1] + list(range(32))), B.SPEC_ERR_INVALID_ARG),      # 33 nodes
])
def test_request_checks(lib, req, expect):
    assert _ws(_req(**req), _attn(), _acc())[0] == expect


def test_null_and_empty_requests(lib):
    dev, host = C.c_size_t(0), C.c_size_t(0)
    assert lib.spec_workspace_bytes(None, None, None, C.byref(dev), C.byref(host)) == B.SPEC_ERR_INVALID_ARG
    r = B.make_requests(np.zeros(0, np.int32), np.zeros(0, np.int32))
    assert _ws(r, _attn(), None)[0] == B.SPEC_ERR_INVALID_ARG
    r = _req()
    r.draft_len = C.POINTER(C.c_int32)()        # chain mode needs draft lengths
    assert _ws(r, _attn(), None)[0] == B.SPEC_ERR_INVALID_ARG


@pytest.mark.parametrize("kw,expect", [
    (dict(num_q_heads=6, num_kv_heads=4), B.SPEC_ERR_INVALID_ARG),
    (dict(num_kv_heads=0), B.SPEC_ERR_INVALID_ARG),
    (dict(head_dim=96), B.SPEC_ERR_UNSUPPORTED),
    (dict(head_dim=64, q_stride_tok=8 * 64, q_stride_head=64, kv_stride_tok=128, kv_stride_head=64), B.SPEC_OK),
    (dict(dtype=7), B.SPEC_ERR_INVALID_ARG),
    (dict(q=None), B.SPEC_ERR_INVALID_ARG),
    (dict(out=None), B.SPEC_ERR_INVALID_ARG),
    (dict(k=FAKE + 2), B.SPEC_ERR_INVALID_ARG),             # misaligned
    (dict(kv_stride_tok=2 * 128 + 4), B.SPEC_ERR_INVALID_ARG),   # bf16 rows must stay 16-byte aligned
    (dict(q_stride_head=0), B.SPEC_ERR_INVALID_ARG),
    (dict(split_kv=33), B.SPEC_ERR_INVALID_ARG),
    (dict(split_kv=-32), B.SPEC_ERR_INVALID_ARG),
    (dict(split_kv=64), B.SPEC_OK),
    (dict(dtype=B.SPEC_F32, kv_stride_tok=2 * 128 + 4), B.SPEC_OK),
])
def test_attention_checks(lib, kw, expect):
    assert _ws(_req(), _attn(**kw), None)[0] == expect


@pytest.mark.parametrize("kw,expect", [
    (dict(vocab=0), B.SPEC_ERR_INVALID_ARG),
    (dict(vocab=4096 * 1024 + 1, logits_stride=4096 * 1024 + 4, probs_stride=4096 * 1024 + 4),
     B.SPEC_ERR_INVALID_ARG),
    (dict(uniforms=None), B.SPEC_ERR_INVALID_ARG),
    (dict(next_token=None), B.SPEC_ERR_INVALID_ARG),
    (dict(draft_tokens=None), B.SPEC_ERR_INVALID_ARG),
    (dict(logits_stride=999), B.SPEC_ERR_INVALID_ARG),
    (dict(logits_stride=1002), B.SPEC_ERR_INVALID_ARG),      # fp32 rows must stay 16-byte aligned
    (dict(dtype=B.SPEC_BF16, logits_stride=1004, probs_stride=1008), B.SPEC_ERR_INVALID_ARG),
    (dict(dtype=B.SPEC_BF16, logits_stride=1008, probs_stride=1008), B.SPEC_OK),
    (dict(target_logits=FAKE + 4), B.SPEC_ERR_INVALID_ARG),
    (dict(dtype=3), B.SPEC_ERR_INVALID_ARG),
    (dict(tree_rule=2), B.SPEC_ERR_INVALID_ARG),
    (dict(tree_rule=B.SPEC_TREE_SEQUENTIAL), B.SPEC_OK),
])
def test_accept_checks(lib, kw, expect):
    assert _ws(_req(), None, _acc(**kw))[0] == expect


def test_all_plain_decoding_needs_no_draft_arrays(lib):
    r = _req(k=(0, 0))
    assert _ws(r, None, _acc(draft_probs=None, draft_tokens=None))[0] == B.SPEC_OK


def test_entry_points_reject_before_any_device_work(lib):
    req, attn, acc = _req(), _attn(), _acc()
    st, dev, host = _ws(req, attn, acc)
    staging = np.full(host + 64, 0xAB, dtype=np.uint8)
    sp = staging.ctypes.data
    # workspace too small / misaligned / missing; staging too small: nothing is written
    assert B.spec_verify(req, attn, acc, FAKE, dev - 256, sp, host, None) == B.SPEC_ERR_WORKSPACE
    assert B.spec_verify(req, attn, acc, FAKE + 64, dev, sp, host, None) == B.SPEC_ERR_WORKSPACE
    assert B.spec_verify(req, attn, acc, 0, dev, sp, host, None) == B.SPEC_ERR_WORKSPACE
    assert B.spec_verify(req, attn, acc, FAKE, dev, sp, host - 1, None) == B.SPEC_ERR_WORKSPACE
    assert B.spec_verify(req, attn, acc, FAKE, dev, 0, host, None) == B.SPEC_ERR_WORKSPACE
    assert (staging == 0xAB).all()
    # missing argument blocks
    assert B.spec_verify(req, None, acc, FAKE, dev, sp, host, None) == B.SPEC_ERR_INVALID_ARG
    assert B.spec_verify(req, attn, None, FAKE, dev, sp, host, None) == B.SPEC_ERR_INVALID_ARG
    assert B.spec_verify_attn(req, None, FAKE, dev, sp, host, None) == B.SPEC_ERR_INVALID_ARG
    assert B.spec_accept(req, None, FAKE, dev, sp, host, None) == B.SPEC_ERR_INVALID_ARG
    # invalid arguments reported by the entry points themselves
    assert B.spec_verify_attn(req, _attn(head_dim=32), FAKE, dev, sp, host, None) == B.SPEC_ERR_UNSUPPORTED
    assert B.spec_accept(_req(k=(1, 99)), acc, FAKE, dev, sp, host, None) == B.SPEC_ERR_INVALID_ARG
    assert (staging == 0xAB).all()


def test_workspace_grows_with_work(lib):
    a = _ws(_req(ctx=(100, 100)), _attn(), _acc())
    b = _ws(_req(ctx=(100, 100, 100, 100), k=(2, 3, 4, 5)), _attn(), _acc())
    c = _ws(_req(), _attn(), _acc(vocab=128256, logits_stride=128256, probs_stride=128256))
    assert a[1] <= b[1] and _ws(_req(), _attn(), _acc())[1] < c[1]


def test_stream_probe_rejects_bad_arguments(lib):
    # every case fails its host check before any HIP call
    assert B.spec_stream_read_probe(0, 1024, FAKE, 64, None) == B.SPEC_ERR_INVALID_ARG
    assert B.spec_stream_read_probe(FAKE + 8, 1024, FAKE, 64, None) == B.SPEC_ERR_INVALID_ARG
    assert B.spec_stream_read_probe(FAKE, 1000, FAKE, 64, None) == B.SPEC_ERR_INVALID_ARG
    assert B.spec_stream_read_probe(FAKE, 0, FAKE, 64, None) == B.SPEC_ERR_INVALID_ARG
    assert B.spec_stream_read_probe(FAKE, 1024, 0, 64, None) == B.SPEC_ERR_INVALID_ARG
    assert B.spec_stream_read_probe(FAKE, 1024, FAKE, 0, None) == B.SPEC_ERR_INVALID_ARG
    assert B.spec_stream_read_probe(FAKE, 1024, FAKE, 65537, None) == B.SPEC_ERR_INVALID_ARG


def test_accept_floor_probe_rejects_bad_arguments(lib):
    # sizes: stream output per (row, chunk), tickets, published values, outputs
    n = B.spec_accept_floor_probe_bytes(32000, 716, 128)
    assert n >= 4 * 716 * 8 + 4 * 128 + 8 * 128 * 8
    assert B.spec_accept_floor_probe_bytes(32000, 100, 128) == 0      # fewer rows than requests
    assert B.spec_accept_floor_probe_bytes(0, 716, 128) == 0
    # every case fails its host check before any HIP call
    ok = (FAKE, 32000, 4, 32000, 716, 128, FAKE, n, FAKE, None)
    def call(**kw):
        args = list(ok)
        for i, k in enumerate(("rows", "stride", "eb", "V", "num_rows", "B", "ws", "ws_bytes", "out", "stream")):
            if k in kw:
                args[i] = kw[k]
        return B.spec_accept_floor_probe(*args)
    assert call(rows=0) == B.SPEC_ERR_INVALID_ARG
    assert call(rows=FAKE + 8) == B.SPEC_ERR_INVALID_ARG
    assert call(ws=0) == B.SPEC_ERR_INVALID_ARG
    assert call(out=0) == B.SPEC_ERR_INVALID_ARG
    assert call(eb=3) == B.SPEC_ERR_INVALID_ARG
    assert call(stride=31999) == B.SPEC_ERR_INVALID_ARG             # shorter than a row
    assert call(stride=32002, eb=2) == B.SPEC_ERR_INVALID_ARG       # rows not 16-byte aligned
    assert call(num_rows=127) == B.SPEC_ERR_INVALID_ARG
    assert call(V=0) == B.SPEC_ERR_INVALID_ARG
    assert call(ws_bytes=n - 1) == B.SPEC_ERR_WORKSPACE


def test_struct_layouts_match_the_header(tmp_path):
    """The ctypes structures of the binding against the C header, field by
    field (offsets and sizes from a program compiled with the system gcc)."""
    import ctypes as C
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("gcc not found")
    structs = {"spec_requests_t": B.SpecRequests, "spec_attn_args_t": B.SpecAttnArgs,
               "spec_accept_args_t": B.SpecAcceptArgs, "spec_sched_params_t": B.SpecSchedParams,
               "spec_sched_state_t": B.SpecSchedState, "spec_sched_request_t": B.SpecSchedRequest,
               "spec_sched_result_t": B.SpecSchedResult}
    lines = ['#include <stdio.h>', '#include <stddef.h>', f'#include "{os.path.join(ROOT, "include", "specsched.h")}"',
             "int main(void) {"]
    for cname, cls in structs.items():
        lines.append(f'  printf("{cname} size %zu\\n", sizeof({cname}));')
        for field, _ in cls._fields_:
            lines.append(f'  printf("{cname} {field} %zu\\n", offsetof({cname}, {field}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", "-o", str(exe), str(src)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out if l.strip()}
    for cname, cls in structs.items():
        assert got[(cname, "size")] == C.sizeof(cls), cname
        for field, _ in cls._fields_:
            assert got[(cname, field)] == getattr(cls, field).offset, (cname, field)


PAGED = dict(block_table=FAKE, block_stride=1, page_tokens=32, num_pages=10)


@pytest.mark.parametrize("kw,expect", [
    (dict(), B.SPEC_OK),                                              # requests of 7 and 12 rows: one page each
    (dict(page_tokens=0), B.SPEC_ERR_INVALID_ARG),
    (dict(page_tokens=16), B.SPEC_ERR_INVALID_ARG),
    (dict(page_tokens=48), B.SPEC_ERR_INVALID_ARG),
    (dict(num_pages=0), B.SPEC_ERR_INVALID_ARG),
    (dict(block_stride=0), B.SPEC_ERR_INVALID_ARG),
    (dict(block_table=FAKE + 2), B.SPEC_ERR_INVALID_ARG),
    (dict(kv_stride_tok=128), B.SPEC_ERR_INVALID_ARG),                # a token row must hold every head
    (dict(dtype=B.SPEC_F32), B.SPEC_ERR_UNSUPPORTED),
    (dict(page_tokens=1 << 23), B.SPEC_ERR_UNSUPPORTED),              # a page beyond 32-bit offsets
])
def test_paged_attention_checks(lib, kw, expect):
    assert _ws(_req(), _attn(**{**PAGED, **kw}), None)[0] == expect


def test_paged_block_stride_must_hold_every_page(lib):
    # 3000 + 3 rows need 94 pages of 32
    assert _ws(_req(ctx=(3000, 5), k=(2, 1)), _attn(**{**PAGED, "block_stride": 93}), None)[0] == B.SPEC_ERR_INVALID_ARG
    assert _ws(_req(ctx=(3000, 5), k=(2, 1)), _attn(**{**PAGED, "block_stride": 94}), None)[0] == B.SPEC_OK


def test_noalloc_checks_before_any_hip_call(lib):
    """spec_verify_noalloc runs the same argument checks as spec_verify before
    any HIP call, and refuses a step that needs more than its static scratch
    (SPEC_ERR_WORKSPACE): both answer on a host without a GPU."""
    h = 0
    assert B.spec_verify_noalloc(_req(ctx=(5, -1)), _attn(), _acc(), h) == B.SPEC_ERR_INVALID_ARG
    assert lib.spec_verify_noalloc(C.byref(_req()), None, C.byref(_acc()), None) == B.SPEC_ERR_INVALID_ARG
    assert lib.spec_verify_noalloc(C.byref(_req()), C.byref(_attn()), None, None) == B.SPEC_ERR_INVALID_ARG
    assert B.spec_verify_noalloc(_req(), _attn(head_dim=96), _acc(), h) == B.SPEC_ERR_UNSUPPORTED
    # 32-key pieces of long contexts: split partials beyond the static scratch
    big = _req(ctx=(60000, 60000, 60000), k=(16, 16, 16))
    st, dev, _ = _ws(big, _attn(split_kv=32), _acc())
    assert st == B.SPEC_OK and dev > B.SPEC_NOALLOC_SCRATCH_BYTES
    assert B.spec_verify_noalloc(big, _attn(split_kv=32), _acc(), h) == B.SPEC_ERR_WORKSPACE
    # the header's limits are the binding's
    text = open(HEADER).read()
    assert "#define SPEC_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)" in text
    assert "#define SPEC_NOALLOC_STAGING_BYTES ((size_t)1 << 20)" in text


def _req_trees(ctx, parents):
    return B.make_requests(np.array(ctx), None, None, tree_parents=parents)


@pytest.mark.parametrize("parents,expect", [
    ([[-1, 0, 0], [-1]], B.SPEC_OK),
    ([[-1, 0, 0], [-1, 0, 1, 1]], B.SPEC_OK),
    ([[-1, 0, 0], [0, 0]], B.SPEC_ERR_INVALID_ARG),          # root's parent must be -1
    ([[-1, 0, 2], [-1]], B.SPEC_ERR_INVALID_ARG),            # parent[n] < n
    ([[-1, 0, 0], [-1] + list(range(32))], B.SPEC_ERR_INVALID_ARG),   # 33 nodes
    ([[-1] + list(range(31)), [-1]], B.SPEC_OK),             # 32 nodes
])
def test_per_request_tree_checks(lib, parents, expect):
    assert _ws(_req_trees([5, 9], parents), _attn(), _acc())[0] == expect


def test_per_request_trees_exclude_a_shared_tree_and_empty_trees(lib):
    r = _req_trees([5, 9], [[-1, 0], [-1]])
    par = np.array([-1, 0], np.int32)
    r.tree_nodes, r.tree_parent = 2, par.ctypes.data_as(C.POINTER(C.c_int32))
    assert _ws(r, _attn(), _acc())[0] == B.SPEC_ERR_INVALID_ARG
    r = _req_trees([5, 9], [[-1, 0], [-1]])
    cnt = np.array([2, 0], np.int32)                           # a request with no node
    r.node_count = cnt.ctypes.data_as(C.POINTER(C.c_int32))
    assert _ws(r, _attn(), _acc())[0] == B.SPEC_ERR_INVALID_ARG
    r = _req_trees([5, 9], [[-1, 0], [-1]])
    r.tree_parents = C.POINTER(C.c_int32)()
    assert _ws(r, _attn(), _acc())[0] == B.SPEC_ERR_INVALID_ARG


def test_per_request_trees_size_like_the_shared_tree(lib):
    """Per-request trees that are all one shared tree need the shared tree's
    device workspace plus the acceptance kernels' copy of the node table, and
    the staged node table (8 bytes per node) on top of the shared plan."""
    tree = [-1, 0, 0, 1, 1, 2, 2]
    ctx = [5, 9, 300]
    shared = _ws(B.make_requests(np.array(ctx), None, tree), _attn(), _acc())
    per = _ws(_req_trees(ctx, [tree] * 3), _attn(), _acc())
    assert shared[0] == per[0] == B.SPEC_OK
    assert per[2] >= shared[2] + 8 * 21 and per[1] >= shared[1] + 8 * 21


def test_claim_word_in_the_workspace(lib, monkeypatch):
    """When the bf16 split kernel has more items than its first round of
    work-groups, the later work-groups claim items from one word in the
    workspace (one more 256-byte section); the fp32 VALU kernel never claims,
    and malformed environment values are ignored."""
    req = _req(ctx=(3000, 5000))
    monkeypatch.setenv("SPEC_ATTN_FIRST_ROUND", str(1 << 20))
    static = _ws(req, _attn(split_kv=1024), None)
    monkeypatch.setenv("SPEC_ATTN_FIRST_ROUND", "1")
    claimed = _ws(req, _attn(split_kv=1024), None)
    monkeypatch.setenv("SPEC_ATTN_EXTRA_WG", "100")          # more work-groups: the same workspace
    assert _ws(req, _attn(split_kv=1024), None) == claimed
    assert static[0] == claimed[0] == B.SPEC_OK and claimed[1] == static[1] + 256
    f32 = dict(dtype=B.SPEC_F32)
    assert _ws(req, _attn(split_kv=1024, **f32), None)[1] == _ws(req, _attn(split_kv=1024, **f32), None)[1]
    monkeypatch.setenv("SPEC_ATTN_FIRST_ROUND", str(1 << 20))
    f32_static = _ws(req, _attn(split_kv=1024, **f32), None)
    monkeypatch.setenv("SPEC_ATTN_FIRST_ROUND", "1")
    assert _ws(req, _attn(split_kv=1024, **f32), None) == f32_static
    for bad in ("0", "-3", "x", "1.5"):                       # ignored: one round of slots
        monkeypatch.setenv("SPEC_ATTN_FIRST_ROUND", bad)
        assert _ws(req, _attn(split_kv=1024), None) == static


def test_fused_combine_counters_in_the_workspace(lib, monkeypatch):
    """Split streams whose partial blocks are under the planner's limit are
    combined inside the bf16 split kernel, which needs one arrival counter per
    split stream in the workspace; the environment limit turns that off, and
    fp32 inputs (the VALU kernel) never use it."""
    req = _req(ctx=(3000, 5000))
    fused = _ws(req, _attn(split_kv=1024), None)           # 16 rows x 5 pieces x 512 B = 40 KB
    monkeypatch.setenv("SPEC_FUSED_COMBINE_MAX_BYTES", "0")
    separate = _ws(req, _attn(split_kv=1024), None)
    monkeypatch.setenv("SPEC_FUSED_COMBINE_MAX_BYTES", "not a number")   # ignored: the default limit
    assert _ws(req, _attn(split_kv=1024), None) == fused
    assert fused[0] == separate[0] == B.SPEC_OK and fused[1] == separate[1] + 256
    monkeypatch.delenv("SPEC_FUSED_COMBINE_MAX_BYTES")
    f32 = dict(dtype=B.SPEC_F32)
    assert _ws(req, _attn(split_kv=1024, **f32), None)[1] == separate[1]
