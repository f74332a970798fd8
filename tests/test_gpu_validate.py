"""The optional device check of the acceptance inputs (SPEC_DEBUG_VALIDATE).

With the environment variable set, spec_accept and spec_verify check the
draft token ids, the uniforms and the draft probability at each draft token
on the device, and return SPEC_ERR_INVALID_ARG before anything that writes an
output is enqueued.  Every case here keeps the bad value inside the arguments'
own buffers, so nothing reads outside them.
"""
import numpy as np
import pytest
import torch

import parity_util as U
from paper_2505_17074_amd import binding as B
from paper_2505_17074_amd.batch import DeviceBatch, Verifier

pytestmark = pytest.mark.gpu

SENTINEL = -7


def _pool():
    return U.custom_pool(ctx=[40, 7, 120], k=[3, 1, 5], Hq=8, Hkv=2, V=3000, seed=11)


def _fill_outputs(b):
    b.accepted_len.fill_(SENTINEL)
    b.next_token.fill_(SENTINEL)
    b.accepted_node.fill_(SENTINEL)
    b.out.fill_(float("nan"))


def _untouched(b, attn=True):
    torch.cuda.synchronize()
    assert (b.accepted_len.cpu().numpy() == SENTINEL).all()
    assert (b.next_token.cpu().numpy() == SENTINEL).all()
    assert (b.accepted_node.cpu().numpy() == SENTINEL).all()
    if attn:
        assert torch.isnan(b.out).all().item()


def test_valid_inputs_pass_and_match(gpu_lib, monkeypatch):
    print("[case] validation on, valid inputs", flush=True)
    pool = _pool()
    b = DeviceBatch(pool, "cuda")
    v = Verifier(b)
    v.run("verify")
    ref = v.results()
    monkeypatch.setenv("SPEC_DEBUG_VALIDATE", "1")
    _fill_outputs(b)
    v.run("verify")
    res = v.results()
    for key in ("accepted_len", "next_token", "accepted_node"):
        np.testing.assert_array_equal(res[key], ref[key])
    np.testing.assert_array_equal(res["out"], ref["out"])


@pytest.mark.parametrize("which", ["accept", "verify"])
@pytest.mark.parametrize("bad", ["token_eq_vocab", "token_negative", "uniform_one", "q_zero_at_token"])
def test_contract_violation_is_reported(gpu_lib, monkeypatch, which, bad):
    print(f"[case] validation on, {bad} via spec_{which}", flush=True)
    pool = _pool()
    b = DeviceBatch(pool, "cuda")
    v = Verifier(b)
    # request 2 (k = 5): its second draft token, and the uniform of that node
    q0 = int(pool.q_start[2])
    t = q0 - 2 + 1                       # token of node 2 (offset n - 1 = 1)
    if bad == "token_eq_vocab":
        b.tokens[t] = pool.vocab
    elif bad == "token_negative":
        b.tokens[t] = -1
    elif bad == "uniform_one":
        b.uniforms[q0 + 2] = 1.0
    else:
        x = int(b.tokens[t].item())
        b.probs[int(pool.d_start[2]) + 1, x] = 0.0     # node 2's parent is node 1 (chain)
    monkeypatch.setenv("SPEC_DEBUG_VALIDATE", "1")
    _fill_outputs(b)
    with pytest.raises(B.SpecError) as e:
        v.run(which)
    assert e.value.status == B.SPEC_ERR_INVALID_ARG
    _untouched(b, attn=(which == "verify"))


def test_unset_or_zero_means_unchecked(gpu_lib, monkeypatch):
    print("[case] validation off ('0')", flush=True)
    pool = _pool()
    b = DeviceBatch(pool, "cuda")
    v = Verifier(b)
    b.uniforms[int(pool.q_start[1])] = 1.0     # outside [0, 1): not checked, no read outside the arguments
    monkeypatch.setenv("SPEC_DEBUG_VALIDATE", "0")
    v.run("accept")
    res = v.results()
    assert (res["accepted_len"] >= 0).all() and (res["next_token"] >= 0).all()


def test_stream_read_probe_reads_every_word(gpu_lib):
    print("[case] stream read probe", flush=True)
    n = (1 << 20) + 48                      # a ragged tail after the eight-load rounds
    src = torch.zeros(n, dtype=torch.uint8, device="cuda")
    src.view(torch.int32)[::7] = 0x5A5A5A5A
    out = torch.empty(1 << 16, dtype=torch.int32, device="cuda")
    for blocks in (1, 3, 64):
        out.zero_()
        B.check(B.spec_stream_read_probe(src.data_ptr(), n, out.data_ptr(), blocks,
                                         torch.cuda.current_stream().cuda_stream), "probe")
        torch.cuda.synchronize()
        # the XOR of every word read, folded over the work-groups, equals the XOR of the buffer
        got = np.bitwise_xor.reduce(out[:blocks].cpu().numpy().view(np.uint32))
        want = np.bitwise_xor.reduce(src.cpu().numpy().view(np.uint32))
        assert got == want, blocks


def _floor_emulated(rows_u8, eb, V, num_rows, B_):
    """The acceptance floor probe's output words, step by step on the host."""
    nch = (V + 4095) // 4096

    def chunk_xor(r, c):
        c0 = c * 4096 * eb
        c1 = min(c0 + 4096 * eb, V * eb)
        n16 = (c1 - c0) // 16
        w = rows_u8[r, c0:c0 + 16 * n16].view(np.uint32)
        return int(np.bitwise_xor.reduce(w)) if w.size else 0

    sink = np.array([[chunk_xor(r, c) for c in range(nch)] for r in range(num_rows)], np.uint64)
    rpr = num_rows // B_
    out = np.zeros(B_, np.uint32)
    for i in range(B_):
        r0 = i * rpr
        x = 0
        for c in range(nch):
            a = int(sink[r0, c])
            b = int(sink[r0 + a % rpr, c])
            x ^= chunk_xor(r0 + b % rpr, c) | 1
        pick = x % nch
        out[i] = chunk_xor(r0 + pick % rpr, pick)
    return out


@pytest.mark.parametrize("eb,V,stride,num_rows,B_", [
    (4, 32000, 32000, 40, 8),       # the LLaMA vocabulary, fp32
    (2, 128256, 128256, 18, 6),     # the long-context vocabulary, bf16
    (4, 5000, 5120, 9, 4),          # a ragged last chunk, padded rows, a row no request owns
])
def test_accept_floor_probe_reads_what_it_claims(gpu_lib, eb, V, stride, num_rows, B_):
    print(f"[case] acceptance floor probe eb {eb} V {V} rows {num_rows} B {B_}", flush=True)
    g = torch.Generator().manual_seed(V + num_rows)
    words = stride * eb // 4
    host = torch.randint(0, 1 << 31, (num_rows, words), dtype=torch.int64, generator=g).to(torch.int32)
    rows = host.to("cuda")
    n = B.spec_accept_floor_probe_bytes(V, num_rows, B_)
    ws = torch.randint(0, 256, (n,), dtype=torch.uint8, device="cuda")       # junk: no initialisation needed
    out = torch.zeros(B_, dtype=torch.int32, device="cuda")
    want = _floor_emulated(host.numpy().view(np.uint8).reshape(num_rows, -1), eb, V, num_rows, B_)
    for _ in range(2):                                                       # the tickets start over each call
        out.fill_(0)
        B.check(B.spec_accept_floor_probe(rows.data_ptr(), stride, eb, V, num_rows, B_, ws.data_ptr(), n,
                                          out.data_ptr(), torch.cuda.current_stream().cuda_stream), "floor probe")
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy().view(np.uint32), want)
