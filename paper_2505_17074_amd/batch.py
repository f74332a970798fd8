"""Packed device batches and a verifier that drives the C ABI.

PyTorch is used for device memory, pinned host memory, streams and events
only; every step of the verify path runs in the library's HIP kernels.
"""
from __future__ import annotations

import ctypes as C
from typing import Optional

import numpy as np
import torch

from . import binding as B
from .workload import BF16, F32, Pool


def _to_device(arr: np.ndarray, dtype: str, device) -> torch.Tensor:
    if dtype == BF16:
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).to(device)
    if dtype == F32:
        return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(device)
    raise ValueError(dtype)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


class DeviceBatch:
    """One verify step's packed inputs and outputs resident in device memory."""

    def __init__(self, pool: Pool, device="cuda"):
        self.pool = pool
        self.device = torch.device(device)
        self.q = _to_device(pool.q, pool.qkv_dtype, self.device)
        self.k = _to_device(pool.k, pool.qkv_dtype, self.device)
        self.v = _to_device(pool.v, pool.qkv_dtype, self.device)
        self.logits = _to_device(pool.target_logits, pool.logit_dtype, self.device)
        self.probs = _to_device(pool.draft_probs, pool.logit_dtype, self.device)
        self.tokens = torch.from_numpy(pool.draft_tokens.astype(np.int32)).to(self.device)
        self.uniforms = torch.from_numpy(pool.uniforms.astype(np.float32)).to(self.device)
        Nq, Hq, d = pool.q.shape
        self.out = torch.empty((Nq, Hq, d), dtype=torch.float32, device=self.device)
        Bn = pool.batch
        self.accepted_len = torch.empty(Bn, dtype=torch.int32, device=self.device)
        self.next_token = torch.empty(Bn, dtype=torch.int32, device=self.device)
        self.accepted_node = torch.empty(Bn, dtype=torch.int32, device=self.device)

    def requests(self) -> B.SpecRequests:
        p = self.pool
        if p.tree_parents is not None:
            return B.make_requests(p.ctx_len, tree_parents=p.tree_parents)
        if p.tree_parent is not None:
            return B.make_requests(p.ctx_len, None, p.tree_parent)
        return B.make_requests(p.ctx_len, p.draft_len)

    def attn_args(self, split_kv: int = 0, scale: float = 0.0) -> B.SpecAttnArgs:
        p = self.pool
        a = B.SpecAttnArgs()
        a.num_q_heads, a.num_kv_heads, a.head_dim = p.num_q_heads, p.num_kv_heads, p.head_dim
        a.dtype = B.SPEC_BF16 if p.qkv_dtype == BF16 else B.SPEC_F32
        a.scale = scale
        a.q, a.k, a.v, a.out = _ptr(self.q), _ptr(self.k), _ptr(self.v), _ptr(self.out)
        a.q_stride_tok, a.q_stride_head = self.q.stride(0), self.q.stride(1)
        a.kv_stride_tok, a.kv_stride_head = self.k.stride(0), self.k.stride(1)
        a.split_kv = split_kv
        return a

    def accept_args(self, with_node: bool = True, tree_rule: int = 0) -> B.SpecAcceptArgs:
        p = self.pool
        a = B.SpecAcceptArgs()
        a.vocab = p.vocab
        a.dtype = B.SPEC_BF16 if p.logit_dtype == BF16 else B.SPEC_F32
        a.target_logits, a.logits_stride = _ptr(self.logits), self.logits.stride(0)
        a.draft_probs = _ptr(self.probs) if self.probs.numel() else None
        a.probs_stride = self.probs.stride(0) if self.probs.numel() else p.vocab
        a.draft_tokens = _ptr(self.tokens) if self.tokens.numel() else None
        a.uniforms = _ptr(self.uniforms)
        a.accepted_len, a.next_token = _ptr(self.accepted_len), _ptr(self.next_token)
        a.accepted_node = _ptr(self.accepted_node) if with_node else None
        a.tree_rule = tree_rule
        return a


class Verifier:
    """Runs spec_verify / spec_verify_attn / spec_accept on one DeviceBatch.

    Owns the device workspace and a ring of `ring` pinned staging buffers,
    one per call in turn.  The slots used since the last event are covered by
    one event, recorded after every `event_every`-th call (and before a call
    on a different stream): each event is a marker packet on the stream, and
    one per call cost the steps 4-7 us.  Before a slot is rewritten, the
    event covering its last use is polled until it completes (a spin, not a
    sleeping wait, so the host never wakes late).  A slot's last use is
    `ring` >= `event_every` calls back, so it is always covered by then.
    Calls may be issued back to back without a device sync.

    Every call uses the one device workspace (split partials, acceptance
    statistics, tickets), so calls are serialised: before a call on a stream
    other than the previous call's, that stream waits on an event recorded
    on the previous call's stream after that call.  Calls that should run
    concurrently need Verifiers of their own.
    """

    def __init__(self, batch: DeviceBatch, split_kv: int = 0, ring: int = 32, event_every: int = 8,
                 attn: Optional[B.SpecAttnArgs] = None):
        if event_every < 1 or ring < event_every:
            raise ValueError("need ring >= event_every >= 1")
        self.batch = batch
        self.req = batch.requests()
        self.attn = attn if attn is not None else batch.attn_args(split_kv)
        self.acc = batch.accept_args()
        st, dev, host = B.spec_workspace_bytes(self.req, self.attn, self.acc)
        B.check(st, "spec_workspace_bytes")
        self.ws_bytes = dev
        self._ws = torch.empty(dev + 256, dtype=torch.uint8, device=batch.device)
        self.ws_ptr = (self._ws.data_ptr() + 255) // 256 * 256
        self.staging_bytes = host
        self._staging = [torch.empty(max(host, 1), dtype=torch.uint8, pin_memory=True) for _ in range(ring)]
        self._every = event_every
        self._slot_ev = [None] * ring      # the event covering each slot's last use
        self._pending = []                 # slots used since the last event
        self._pending_stream = None
        self._i = 0                        # calls issued
        self._last_stream = None           # stream of the previous call (workspace owner)

    def _order(self, stream):
        """Make `stream` wait for the previous call when that call ran on
        another stream: the two share the workspace."""
        last = self._last_stream
        if last is not None and stream != last:
            ev = torch.cuda.Event()
            ev.record(last)
            stream.wait_event(ev)
        self._last_stream = stream

    def _cover(self):
        # a new event each time: one recorded again later, perhaps on another
        # stream, would no longer order the slots that still hold it
        if self._pending:
            ev = torch.cuda.Event()
            ev.record(self._pending_stream)
            for s in self._pending:
                self._slot_ev[s] = ev
            self._pending = []

    def _slot(self, stream):
        if self._pending and stream != self._pending_stream:
            self._cover()
        s = self._i % len(self._staging)
        ev = self._slot_ev[s]              # never pending: fewer than event_every <= ring calls are
        if ev is not None:
            while not ev.query():
                pass
        self._i += 1
        return s

    def _done(self, s, stream):
        self._slot_ev[s] = None
        self._pending.append(s)
        self._pending_stream = stream
        if len(self._pending) >= self._every:
            self._cover()

    def run(self, which: str = "verify", stream: Optional[torch.cuda.Stream] = None) -> None:
        stream = stream or torch.cuda.current_stream(self.batch.device)
        s = self._slot(stream)
        self._order(stream)
        stg = self._staging[s].data_ptr()
        h = stream.cuda_stream
        try:
            if which == "verify":
                st = B.spec_verify(self.req, self.attn, self.acc, self.ws_ptr, self.ws_bytes, stg, self.staging_bytes, h)
            elif which == "attn":
                st = B.spec_verify_attn(self.req, self.attn, self.ws_ptr, self.ws_bytes, stg, self.staging_bytes, h)
            elif which == "accept":
                st = B.spec_accept(self.req, self.acc, self.ws_ptr, self.ws_bytes, stg, self.staging_bytes, h)
            else:
                raise ValueError(which)
        finally:
            self._done(s, stream)       # a failed call's slot is covered like any other
        B.check(st, f"spec_{which}")

    def results(self) -> dict:
        torch.cuda.synchronize(self.batch.device)
        b = self.batch
        return {"out": b.out.cpu().numpy(),
                "accepted_len": b.accepted_len.cpu().numpy(),
                "next_token": b.next_token.cpu().numpy(),
                "accepted_node": b.accepted_node.cpu().numpy()}


class PagedKV:
    """A DeviceBatch's K/V rows in page pools [num_pages, page_tokens, Hkv, d]
    (the paged layout of specverify.h), pages in a seeded random order with
    `spare` unused pages in between, and the block table [B, block_stride].
    Rows past a request's length in its last page are zero.  `attn_args`
    returns attention arguments that read the pools through the table."""

    def __init__(self, batch: DeviceBatch, page_tokens: int = 64, seed: int = 0, spare: int = 3):
        pool = batch.pool
        P = int(page_tokens)
        L = (pool.ctx_len.astype(np.int64) + pool.n_q.astype(np.int64))
        pages = (L + P - 1) // P
        total = int(pages.sum())
        self.page_tokens, self.num_pages = P, total + int(spare)
        self.block_stride = int(pages.max())
        rng = np.random.default_rng(seed)
        order = rng.permutation(self.num_pages)[:total].astype(np.int32)
        table = np.zeros((pool.batch, self.block_stride), np.int32)
        start = np.concatenate([[0], np.cumsum(pages)])
        src, dst = [], []
        kv0 = np.concatenate([[0], np.cumsum(L)])
        for i in range(pool.batch):
            table[i, :pages[i]] = order[start[i]:start[i + 1]]
            t = np.arange(L[i])
            src.append(kv0[i] + t)
            dst.append(table[i, t // P].astype(np.int64) * P + t % P)
        src = torch.from_numpy(np.concatenate(src)).to(batch.device)
        dst = torch.from_numpy(np.concatenate(dst)).to(batch.device)
        Hkv, d = batch.k.shape[1], batch.k.shape[2]
        self.k = torch.zeros((self.num_pages * P, Hkv, d), dtype=batch.k.dtype, device=batch.device)
        self.v = torch.zeros_like(self.k)
        self.k[dst] = batch.k[src]
        self.v[dst] = batch.v[src]
        self.table = torch.from_numpy(table).to(batch.device)
        self.table_np = table
        self.batch = batch

    def attn_args(self, split_kv: int = 0, scale: float = 0.0) -> B.SpecAttnArgs:
        a = self.batch.attn_args(split_kv, scale)
        a.k, a.v = self.k.data_ptr(), self.v.data_ptr()
        a.kv_stride_tok, a.kv_stride_head = self.k.stride(0), self.k.stride(1)
        a.block_table = self.table.data_ptr()
        a.block_stride, a.page_tokens, a.num_pages = self.block_stride, self.page_tokens, self.num_pages
        return a


def pad_vocab_rows(batch: DeviceBatch) -> None:
    """Give the batch's logits and draft rows a row stride padded to 16 bytes
    (the ABI's row alignment), whatever the vocabulary size."""
    for attr in ("logits", "probs"):
        t = getattr(batch, attr)
        vec = 16 // t.element_size()
        V = t.shape[1]
        Vp = -(-V // vec) * vec
        if Vp != V and t.numel():
            pad = torch.zeros((t.shape[0], Vp), dtype=t.dtype, device=batch.device)
            pad[:, :V] = t
            setattr(batch, attr, pad[:, :V])


class LmHeadVerifier:
    """spec_lm_head_accept on a pool from workload.make_lm_head_pool: the
    hidden states and LM-head weights in device memory, the logits buffer
    the GEMM writes (then read by the acceptance), the draft inputs and the
    outputs; a device workspace and one pinned staging buffer (each call
    waits for the previous one before rewriting it)."""

    def __init__(self, pool: Pool, device="cuda"):
        if pool.hidden is None or pool.weight is None:
            raise ValueError("the pool carries no LM-head inputs")
        self.batch = DeviceBatch(pool, device)        # logits buffer (zeros), draft rows, tokens, uniforms, outputs
        dev = self.batch.device
        pad_vocab_rows(self.batch)
        self.hidden = torch.from_numpy(np.ascontiguousarray(pool.hidden).view(np.int16)).view(torch.bfloat16).to(dev)
        self.weight = torch.from_numpy(np.ascontiguousarray(pool.weight).view(np.int16)).view(torch.bfloat16).to(dev)
        self.req = self.batch.requests()
        self.lm = B.SpecLmHeadArgs()
        self.lm.hidden_dim = int(pool.hidden.shape[1])
        self.lm.hidden, self.lm.hidden_stride = self.hidden.data_ptr(), self.hidden.stride(0)
        self.lm.weight, self.lm.weight_stride = self.weight.data_ptr(), self.weight.stride(0)
        self.acc = self.batch.accept_args()
        st, dbytes, hbytes = B.spec_lm_head_workspace_bytes(self.req, self.lm, self.acc)
        B.check(st, "spec_lm_head_workspace_bytes")
        self.ws_bytes = dbytes
        self._ws = torch.empty(dbytes + 256, dtype=torch.uint8, device=dev)
        self.ws_ptr = (self._ws.data_ptr() + 255) // 256 * 256
        self.staging_bytes = hbytes
        self._staging = torch.empty(max(hbytes, 1), dtype=torch.uint8, pin_memory=True)
        self._done = None

    def run(self, stream: Optional[torch.cuda.Stream] = None) -> None:
        stream = stream or torch.cuda.current_stream(self.batch.device)
        if self._done is not None:
            self._done.synchronize()      # the staging buffer is rewritten by this call
        st = B.spec_lm_head_accept(self.req, self.lm, self.acc, self.ws_ptr, self.ws_bytes,
                                   self._staging.data_ptr(), self.staging_bytes, stream.cuda_stream)
        self._done = torch.cuda.Event()
        self._done.record(stream)
        B.check(st, "spec_lm_head_accept")

    def logits(self) -> np.ndarray:
        """The logits the GEMM wrote, in their storage format."""
        torch.cuda.synchronize(self.batch.device)
        t = self.batch.logits.contiguous()
        return t.view(torch.int16).cpu().numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.cpu().numpy()

    def results(self) -> dict:
        torch.cuda.synchronize(self.batch.device)
        b = self.batch
        return {"accepted_len": b.accepted_len.cpu().numpy(), "next_token": b.next_token.cpu().numpy(),
                "accepted_node": b.accepted_node.cpu().numpy()}
