"""Python-side handles over the C ABI: device memory comes from torch (HIP
allocations on the current device), every computation from libdash.so.

    model = Model(shape, weights)                 # uploads weights, dash_model_create
    kv = KVCache(model, page_size, max_seqs, max_ctx, n_pages)
    toks, lps = rollout(model, kv, prompts, group, gen_len)
    adv, kept = advantage_filter(rewards, group)
"""
from __future__ import annotations

import numpy as np
import torch

from . import _lib as L
from . import synth


def stream_handle() -> int:
    return torch.cuda.current_stream().cuda_stream


def _to_device(arr: np.ndarray, dtype_code: int, device) -> torch.Tensor:
    if dtype_code == L.DASH_BF16:
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(device)


def desc_of(shape: synth.Shape) -> L.dash_model_desc:
    return L.dash_model_desc(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim,
                             shape.d_ff, shape.vocab, shape.dtype, shape.rope_theta, shape.rms_eps)


class Model:
    """Device weights (torch tensors, caller-owned from the library's view) + dash_model handle."""

    def __init__(self, shape: synth.Shape, weights: dict, device: str = "cuda"):
        self.shape = shape
        self.device = torch.device(device)
        self.tensors = {}
        ptrs = []
        for name in synth.weight_names(shape):
            arr = weights[name]
            if arr.size == 0:
                ptrs.append(None)
                continue
            t = _to_device(arr, shape.dtype, self.device)
            self.tensors[name] = t
            ptrs.append(t.data_ptr())
        self.desc = desc_of(shape)
        self.handle = L.dash_model_create(self.desc, ptrs)

    def close(self):
        if getattr(self, "handle", None):
            L.dash_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def workspace(self, max_rows: int, max_ctx: int = 0) -> torch.Tensor:
        n = L.dash_workspace_bytes(self.handle, max_rows, max_ctx)
        return torch.empty(n + 256, dtype=torch.uint8, device=self.device)


class KVCache:
    """Paged KV pool + page table (torch device buffers) and the dash_kv handle."""

    def __init__(self, model: Model, page_size: int, max_seqs: int, max_ctx: int, n_pages: int):
        self.model = model
        self.page_size = page_size
        self.max_seqs, self.max_ctx = max_seqs, max_ctx
        page_bytes = L.dash_kv_page_bytes(model.handle, page_size)
        # zero-filled once: positions never written read as zeros, not as stale bits
        self.pool = torch.zeros(n_pages * page_bytes, dtype=torch.uint8, device=model.device)
        tb = L.dash_kv_table_bytes(max_seqs, max_ctx, page_size)
        self.table = torch.empty(tb, dtype=torch.uint8, device=model.device)
        self.handle = L.dash_kv_create(model.handle, self.pool.data_ptr(), self.pool.numel(), page_size, max_seqs,
                                       max_ctx, self.table.data_ptr(), stream_handle())

    @property
    def free_pages(self) -> int:
        return L.dash_kv_free_pages(self.handle)

    @property
    def split_keys(self) -> int:
        return L.dash_kv_split_keys(self.handle)

    def close(self):
        if getattr(self, "handle", None):
            torch.cuda.synchronize()
            L.dash_kv_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def aligned(buf: torch.Tensor) -> int:
    """256-byte aligned device address inside `buf` (allocated with 256 spare bytes)."""
    p = buf.data_ptr()
    return (p + 255) // 256 * 256


def prefill(model: Model, kv: KVCache, prompts: torch.Tensor, group: int, slots, ws: torch.Tensor | None = None):
    """dash_prefill: returns float32 logits [n_prompts, vocab]."""
    n_prompts, P = prompts.shape
    logits = torch.empty(n_prompts, model.shape.vocab, dtype=torch.float32, device=model.device)
    if ws is None:
        ws = model.workspace(n_prompts * P, 0)
    L.dash_prefill(model.handle, kv.handle, prompts.data_ptr(), n_prompts, P, group, list(slots), logits.data_ptr(),
                   aligned(ws), ws.numel() - 256, stream_handle())
    return logits


def decode_step(model: Model, kv: KVCache, tokens: torch.Tensor, slots: torch.Tensor, pos: torch.Tensor,
                ws: torch.Tensor | None = None, logits: torch.Tensor | None = None):
    """dash_decode_step: returns float32 logits [n_rows, vocab]."""
    n = tokens.numel()
    if logits is None:
        logits = torch.empty(n, model.shape.vocab, dtype=torch.float32, device=model.device)
    if ws is None:
        ws = model.workspace(n, kv.max_ctx)
    L.dash_decode_step(model.handle, kv.handle, tokens.data_ptr(), slots.data_ptr(), pos.data_ptr(), n,
                       logits.data_ptr(), aligned(ws), ws.numel() - 256, stream_handle())
    return logits


def decode_step_grouped(model: Model, kv: KVCache, tokens: torch.Tensor, slots: torch.Tensor, pos: torch.Tensor,
                        group_off: torch.Tensor, group_size: int, shared_len: int, ws: torch.Tensor | None = None,
                        logits: torch.Tensor | None = None):
    """dash_decode_step_grouped: rows [group_off[i], group_off[i+1]) share their first shared_len positions."""
    n = tokens.numel()
    if logits is None:
        logits = torch.empty(n, model.shape.vocab, dtype=torch.float32, device=model.device)
    if ws is None:
        ws = model.workspace(n, kv.max_ctx)
    L.dash_decode_step_grouped(model.handle, kv.handle, tokens.data_ptr(), slots.data_ptr(), pos.data_ptr(), n,
                               group_off.data_ptr(), group_off.numel() - 1, group_size, shared_len,
                               logits.data_ptr(), aligned(ws), ws.numel() - 256, stream_handle())
    return logits


def sample(logits: torch.Tensor, seq_uid: torch.Tensor, step: torch.Tensor, temperature: float, seed: int,
           row_of: torch.Tensor | None = None, n_rows: int | None = None, with_logprob: bool = True,
           row_max_lse: torch.Tensor | None = None, status: torch.Tensor | None = None):
    """dash_sample: returns (int32 tokens [n_rows], float32 logprobs [n_rows] or None).
    Optional outputs: row_max_lse float32 [n_rows, 2]; status uint32/int32 [1] (bits OR-ed in)."""
    n = seq_uid.numel() if n_rows is None else n_rows
    V = logits.shape[-1]
    toks = torch.empty(n, dtype=torch.int32, device=logits.device)
    lps = torch.empty(n, dtype=torch.float32, device=logits.device) if with_logprob else None
    L.dash_sample(logits.data_ptr(), logits.stride(0), n, V, L.ptr(row_of), seq_uid.data_ptr(), step.data_ptr(),
                  temperature, seed, toks.data_ptr(), L.ptr(lps), L.ptr(row_max_lse), L.ptr(status), stream_handle())
    return toks, lps


def advantage_filter(rewards: torch.Tensor, group: int, mode: int = L.DASH_ADV_STD_SAMPLE, eps: float = 1e-6,
                     tau: float = 0.1):
    """dash_group_advantage_filter: returns (float32 A [N], int32 kept indices [K] on the device)."""
    N = rewards.numel()
    adv = torch.empty(N, dtype=torch.float32, device=rewards.device)
    kept = torch.empty(N, dtype=torch.int32, device=rewards.device)
    cnt = torch.empty(1, dtype=torch.int32, device=rewards.device)
    L.dash_group_advantage_filter(rewards.data_ptr(), N // group, group, mode, eps, tau, adv.data_ptr(),
                                  kept.data_ptr(), cnt.data_ptr(), stream_handle())
    k = int(cnt.item())
    return adv, kept[:k]


def teacher_forced_logprobs(model: Model, kv: KVCache, seqs: torch.Tensor, prompt_len: int,
                            seqs_per_chunk: int = 8) -> torch.Tensor:
    """dash_teacher_forced_logprobs: int32 [n, L] (prompt + completion) -> float32 [n, L - prompt_len]."""
    n, Ls = seqs.shape
    out = torch.empty((n, Ls - prompt_len), dtype=torch.float32, device=seqs.device)
    c = max(1, min(seqs_per_chunk, n))
    nbytes = L.dash_teacher_forced_workspace_bytes(model.handle, c, Ls, prompt_len)
    ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=seqs.device)
    L.dash_teacher_forced_logprobs(model.handle, kv.handle, seqs.data_ptr(), n, Ls, prompt_len, out.data_ptr(),
                                   aligned(ws), nbytes, stream_handle())
    return out


def pg_loss(logprobs: torch.Tensor, adv: torch.Tensor, kept: torch.Tensor, lengths: torch.Tensor | None = None):
    """dash_pg_loss over the kept indices: returns (float64 loss [1], float64 sequence log-probs [N])."""
    N, T = logprobs.shape
    dev = logprobs.device
    cnt = torch.tensor([kept.numel()], dtype=torch.int32, device=dev)
    loss = torch.empty(1, dtype=torch.float64, device=dev)
    seq = torch.zeros(N, dtype=torch.float64, device=dev)
    kept_buf = kept if kept.numel() else torch.zeros(1, dtype=torch.int32, device=dev)
    L.dash_pg_loss(logprobs.data_ptr(), logprobs.stride(0), T, lengths.data_ptr() if lengths is not None else None,
                   adv.data_ptr(), kept_buf.data_ptr(), cnt.data_ptr(), N, loss.data_ptr(), seq.data_ptr(),
                   stream_handle())
    return loss, seq


def policy_loss(logprobs: torch.Tensor, adv: torch.Tensor, kept: torch.Tensor, lengths: torch.Tensor | None = None,
                logprobs_old: torch.Tensor | None = None, kl: torch.Tensor | None = None, clip_eps: float = 0.2,
                beta: float = 0.0):
    """dash_policy_loss: (float64 loss [1], float64 stats [N, 4] = (S, S_old, KL, d loss / d S) per kept sample)."""
    N, T = logprobs.shape
    dev = logprobs.device
    for t in (logprobs_old, kl):
        if t is not None and (t.shape != logprobs.shape or t.stride() != logprobs.stride()):
            raise ValueError("logprobs_old and kl must have the logprobs' shape and strides")
    cnt = torch.tensor([kept.numel()], dtype=torch.int32, device=dev)
    loss = torch.empty(1, dtype=torch.float64, device=dev)
    stats = torch.zeros(N, 4, dtype=torch.float64, device=dev)
    kept_buf = kept if kept.numel() else torch.zeros(1, dtype=torch.int32, device=dev)
    L.dash_policy_loss(logprobs.data_ptr(), logprobs_old.data_ptr() if logprobs_old is not None else None,
                       kl.data_ptr() if kl is not None else None, logprobs.stride(0), T,
                       lengths.data_ptr() if lengths is not None else None, adv.data_ptr(), kept_buf.data_ptr(),
                       cnt.data_ptr(), N, clip_eps, beta, loss.data_ptr(), stats.data_ptr(), stream_handle())
    return loss, stats


def logits_kl(theta: torch.Tensor, base: torch.Tensor, reverse: bool = True):
    """dash_logits_kl on float32 [rows, V] logits: (D_KL(base || theta) [rows], D_KL(theta || base) [rows] or None)."""
    if theta.shape != base.shape or theta.stride() != base.stride() or theta.dim() != 2:
        raise ValueError("theta and base logits must be 2-D with equal shapes and strides")
    rows, V = theta.shape
    kl = torch.empty(rows, dtype=torch.float32, device=theta.device)
    kl_rev = torch.empty(rows, dtype=torch.float32, device=theta.device) if reverse else None
    L.dash_logits_kl(theta.data_ptr(), base.data_ptr(), theta.stride(0), rows, V, kl.data_ptr(),
                     kl_rev.data_ptr() if kl_rev is not None else None, stream_handle())
    return kl, kl_rev


def teacher_forced_kl(model: Model, base: Model, kv: KVCache, seqs: torch.Tensor, prompt_len: int,
                      seqs_per_chunk: int = 8, with_logprobs: bool = True, reverse: bool = True):
    """dash_teacher_forced_kl: int32 [n, L] -> (log-probs or None, KL(base || policy), KL(policy || base) or None),
    each float32 [n, L - prompt_len]."""
    n, Ls = seqs.shape
    shp = (n, Ls - prompt_len)
    lp = torch.empty(shp, dtype=torch.float32, device=seqs.device) if with_logprobs else None
    kl = torch.empty(shp, dtype=torch.float32, device=seqs.device)
    kl_rev = torch.empty(shp, dtype=torch.float32, device=seqs.device) if reverse else None
    c = max(1, min(seqs_per_chunk, n))
    nbytes = L.dash_teacher_forced_kl_workspace_bytes(model.handle, c, Ls, prompt_len)
    ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=seqs.device)
    L.dash_teacher_forced_kl(model.handle, base.handle, kv.handle, seqs.data_ptr(), n, Ls, prompt_len,
                             lp.data_ptr() if lp is not None else None, kl.data_ptr(),
                             kl_rev.data_ptr() if kl_rev is not None else None, aligned(ws), nbytes, stream_handle())
    return lp, kl, kl_rev


class Rollout:
    """Reusable buffers for dash_rollout on one workload shape."""

    def __init__(self, model: Model, kv: KVCache, n_prompts: int, prompt_len: int, group: int, gen_len: int):
        self.model, self.kv = model, kv
        self.n_prompts, self.P, self.G, self.T = n_prompts, prompt_len, group, gen_len
        N = n_prompts * group
        n = L.dash_rollout_workspace_bytes(model.handle, n_prompts, prompt_len, group, kv.max_ctx)
        self.ws = torch.empty(n + 256, dtype=torch.uint8, device=model.device)
        self.tokens = torch.empty(N, gen_len, dtype=torch.int32, device=model.device)
        self.logprobs = torch.empty(N, gen_len, dtype=torch.float32, device=model.device)
        # HIP graphs cannot be captured on the legacy null stream: run on a side
        # stream (default priority) ordered against the caller's stream.
        self.stream = torch.cuda.Stream(device=model.device)

    def run(self, prompts: torch.Tensor, temperature: float = 1.0, seed: int = 2, budgets=None,
            use_graph: bool = True, with_logprobs: bool = True):
        cur = torch.cuda.current_stream(self.model.device)
        self.stream.wait_stream(cur)
        L.dash_rollout(self.model.handle, self.kv.handle, prompts.data_ptr(), self.n_prompts, self.P, self.G, self.T,
                       budgets, temperature, seed, self.tokens.data_ptr(),
                       self.logprobs.data_ptr() if with_logprobs else None, use_graph, aligned(self.ws),
                       self.ws.numel() - 256, self.stream.cuda_stream)
        cur.wait_stream(self.stream)
        return self.tokens, self.logprobs
