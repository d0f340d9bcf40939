"""ctypes binding of libdash.so (include/dash.h): the same function names, argument
marshalling only.  Every computation happens inside the library's HIP kernels.

The library is loaded from this package directory; if it is missing the import
of any compute entry point raises — there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdash.so")

DASH_OK, DASH_EINVAL, DASH_ENOMEM, DASH_ECAPACITY, DASH_EDEVICE, DASH_ENOTSUP = range(6)
# device status bits (dash_kv_device_status, dash_sample's status word)
DASH_ST_UNBACKED, DASH_ST_NO_FINITE_LOGIT, DASH_ST_BAD_TOKEN = 1, 2, 4
DASH_F32, DASH_BF16 = 0, 1
DASH_ADV_MEAN_ONLY, DASH_ADV_STD_POP, DASH_ADV_STD_SAMPLE, DASH_ADV_LOO = 0, 1, 2, 3
K_CLASSES = ["prefill", "embed", "norm", "rope", "gemm_qkv", "attn", "attn_combine", "gemm_o", "gemm_gate_up",
             "gemm_down", "gemm_lm_head", "sample", "advantage", "other"]
K = {name: i for i, name in enumerate(K_CLASSES)}


class DashError(RuntimeError):
    def __init__(self, status: int, func: str, text: str):
        super().__init__(f"{func}: status {status} ({_status_names.get(status, '?')}): {text}")
        self.status = status


_status_names = {0: "DASH_OK", 1: "DASH_EINVAL", 2: "DASH_ENOMEM", 3: "DASH_ECAPACITY", 4: "DASH_EDEVICE",
                 5: "DASH_ENOTSUP"}


class dash_model_desc(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("d_ff", C.c_int32),
                ("vocab", C.c_int32), ("dtype", C.c_int32), ("rope_theta", C.c_float), ("rms_eps", C.c_float)]


_P = C.c_void_p
_I32P = C.POINTER(C.c_int32)
_SIGS = {
    "dash_abi_version": (C.c_int, []),
    "dash_status_str": (C.c_char_p, [C.c_int]),
    "dash_last_error": (C.c_char_p, []),
    "dash_weight_count": (C.c_int32, [C.POINTER(dash_model_desc)]),
    "dash_model_create": (C.c_int, [C.POINTER(dash_model_desc), C.POINTER(_P), C.c_int32, C.POINTER(_P)]),
    "dash_model_destroy": (None, [_P]),
    "dash_kv_page_bytes": (C.c_size_t, [_P, C.c_int32]),
    "dash_kv_table_bytes": (C.c_size_t, [C.c_int32, C.c_int32, C.c_int32]),
    "dash_kv_create": (C.c_int, [_P, _P, C.c_size_t, C.c_int32, C.c_int32, C.c_int32, _P, _P, C.POINTER(_P)]),
    "dash_kv_destroy": (None, [_P]),
    "dash_kv_free_pages": (C.c_int, [_P, _I32P]),
    "dash_kv_slot_len": (C.c_int, [_P, C.c_int32, _I32P]),
    "dash_kv_split_keys": (C.c_int, [_P, _I32P]),
    "dash_kv_reserve": (C.c_int, [_P, _I32P, C.c_int32, C.c_int32, _P]),
    "dash_kv_release": (C.c_int, [_P, _I32P, C.c_int32]),
    "dash_kv_device_status": (C.c_int, [_P, C.POINTER(C.c_uint32), _P]),
    "dash_workspace_bytes": (C.c_size_t, [_P, C.c_int32, C.c_int32]),
    "dash_prefill": (C.c_int, [_P, _P, _P, C.c_int32, C.c_int32, C.c_int32, _I32P, _P, _P, C.c_size_t, _P]),
    "dash_decode_step": (C.c_int, [_P, _P, _P, _P, _P, C.c_int32, _P, _P, C.c_size_t, _P]),
    "dash_decode_step_noalloc": (C.c_int, [_P, _P, _P, _P, _P, C.c_int32, _P, _P]),
    "dash_decode_step_grouped": (C.c_int, [_P, _P, _P, _P, _P, C.c_int32, _P, C.c_int32, C.c_int32, C.c_int32, _P,
                                           _P, C.c_size_t, _P]),
    "dash_sample": (C.c_int, [_P, C.c_int64, C.c_int32, C.c_int32, _P, _P, _P, C.c_float, C.c_uint64, _P, _P, _P,
                              _P, _P]),
    "dash_sampler_check": (C.c_int, [C.POINTER(C.c_double), C.POINTER(C.c_double)]),
    "dash_bf16_round_check": (C.c_int, [C.POINTER(C.c_uint64)]),
    "dash_group_advantage_filter": (C.c_int, [_P, C.c_int32, C.c_int32, C.c_int32, C.c_float, C.c_float, _P, _P,
                                              _P, _P]),
    "dash_live_compact": (C.c_int, [_P, _P, _P, _P, _P, _P, C.c_int32, C.c_int32, _P, _P, _P, _P, _P, _P, _P]),
    "dash_teacher_forced_workspace_bytes": (C.c_size_t, [_P, C.c_int32, C.c_int32, C.c_int32]),
    "dash_teacher_forced_logprobs": (C.c_int, [_P, _P, _P, C.c_int32, C.c_int32, C.c_int32, _P, _P, C.c_size_t, _P]),
    "dash_pg_loss": (C.c_int, [_P, C.c_int64, C.c_int32, _P, _P, _P, _P, C.c_int32, _P, _P, _P]),
    "dash_policy_loss": (C.c_int, [_P, _P, _P, C.c_int64, C.c_int32, _P, _P, _P, _P, C.c_int32, C.c_double,
                                   C.c_double, _P, _P, _P]),
    "dash_logits_kl": (C.c_int, [_P, _P, C.c_int64, C.c_int32, C.c_int32, _P, _P, _P]),
    "dash_teacher_forced_kl_workspace_bytes": (C.c_size_t, [_P, C.c_int32, C.c_int32, C.c_int32]),
    "dash_teacher_forced_kl": (C.c_int, [_P, _P, _P, _P, C.c_int32, C.c_int32, C.c_int32, _P, _P, _P, _P,
                                         C.c_size_t, _P]),
    "dash_rollout_workspace_bytes": (C.c_size_t, [_P, C.c_int32, C.c_int32, C.c_int32, C.c_int32]),
    "dash_rollout": (C.c_int, [_P, _P, _P, C.c_int32, C.c_int32, C.c_int32, C.c_int32, _I32P, C.c_float, C.c_uint64,
                               _P, _P, C.c_int32, _P, C.c_size_t, _P]),
    "dash_profile_enable": (C.c_int, [C.c_uint32]),
    "dash_profile_layer": (C.c_int, [C.c_int32]),
    "dash_profile_read": (C.c_int, [C.POINTER(C.c_double), C.POINTER(C.c_int64), C.c_int32]),
}

_lib = None


def load() -> C.CDLL:
    """Load libdash.so; raise FileNotFoundError if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise FileNotFoundError(f"{LIB_PATH} is missing: build it with `python -m paper_2505_17218_amd.build`")
        lib = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(lib, name)
            f.restype = res
            f.argtypes = args
        _lib = lib
    return _lib


def header_functions() -> list[str]:
    return list(_SIGS)


def check(status: int, func: str) -> None:
    if status != DASH_OK:
        raise DashError(status, func, load().dash_last_error().decode())


def _call(name: str, *args) -> int:
    st = getattr(load(), name)(*args)
    check(st, name)
    return st


def ptr(t) -> int | None:
    """Device pointer of a torch tensor (or None / int passthrough)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def i32_array(vals) -> C.Array:
    vals = [int(v) for v in vals]
    return (C.c_int32 * max(1, len(vals)))(*vals)


# ---- thin wrappers with the C names ----------------------------------------

def dash_abi_version() -> int:
    return load().dash_abi_version()


def dash_weight_count(desc: dash_model_desc) -> int:
    return load().dash_weight_count(C.byref(desc))


def dash_model_create(desc: dash_model_desc, weight_ptrs: list) -> int:
    arr = (_P * len(weight_ptrs))(*[p if p else None for p in weight_ptrs])
    out = _P()
    _call("dash_model_create", C.byref(desc), arr, len(weight_ptrs), C.byref(out))
    return out.value


def dash_model_destroy(h: int) -> None:
    load().dash_model_destroy(h)


def dash_kv_page_bytes(model: int, page_size: int) -> int:
    return load().dash_kv_page_bytes(model, page_size)


def dash_kv_table_bytes(max_seqs: int, max_ctx: int, page_size: int) -> int:
    return load().dash_kv_table_bytes(max_seqs, max_ctx, page_size)


def dash_kv_create(model: int, pool: int, pool_bytes: int, page_size: int, max_seqs: int, max_ctx: int,
                   table: int, stream: int | None) -> int:
    out = _P()
    _call("dash_kv_create", model, pool, pool_bytes, page_size, max_seqs, max_ctx, table, stream, C.byref(out))
    return out.value


def dash_kv_destroy(h: int) -> None:
    load().dash_kv_destroy(h)


def dash_kv_free_pages(kv: int) -> int:
    out = C.c_int32()
    _call("dash_kv_free_pages", kv, C.byref(out))
    return out.value


def dash_kv_slot_len(kv: int, slot: int) -> int:
    out = C.c_int32()
    _call("dash_kv_slot_len", kv, slot, C.byref(out))
    return out.value


def dash_kv_split_keys(kv: int) -> int:
    out = C.c_int32()
    _call("dash_kv_split_keys", kv, C.byref(out))
    return out.value


def dash_kv_reserve(kv: int, slots, new_len: int, stream: int | None) -> None:
    _call("dash_kv_reserve", kv, i32_array(slots), len(slots), new_len, stream)


def dash_kv_release(kv: int, slots) -> None:
    _call("dash_kv_release", kv, i32_array(slots), len(slots))


def dash_kv_device_status(kv: int, stream: int | None) -> int:
    out = C.c_uint32()
    _call("dash_kv_device_status", kv, C.byref(out), stream)
    return out.value


def dash_workspace_bytes(model: int, max_rows: int, max_ctx: int) -> int:
    return load().dash_workspace_bytes(model, max_rows, max_ctx)


def dash_prefill(model, kv, d_tokens, n_prompts, prompt_len, group, slots, d_logits, d_ws, ws_bytes, stream):
    _call("dash_prefill", model, kv, d_tokens, n_prompts, prompt_len, group, i32_array(slots), d_logits, d_ws,
          ws_bytes, stream)


def dash_decode_step(model, kv, d_tokens, d_slots, d_pos, n_rows, d_logits, d_ws, ws_bytes, stream):
    _call("dash_decode_step", model, kv, d_tokens, d_slots, d_pos, n_rows, d_logits, d_ws, ws_bytes, stream)


def dash_decode_step_noalloc(model, kv, d_tokens, d_slots, d_pos, n_rows, d_logits, stream):
    _call("dash_decode_step_noalloc", model, kv, d_tokens, d_slots, d_pos, n_rows, d_logits, stream)


def dash_decode_step_grouped(model, kv, d_tokens, d_slots, d_pos, n_rows, d_group_off, n_groups, group_size,
                             shared_len, d_logits, d_ws, ws_bytes, stream):
    _call("dash_decode_step_grouped", model, kv, d_tokens, d_slots, d_pos, n_rows, d_group_off, n_groups, group_size,
          shared_len, d_logits, d_ws, ws_bytes, stream)


def dash_sample(d_logits, ld, n_rows, vocab, d_row_of, d_seq_uid, d_step, temperature, seed, d_tokens_out,
                d_logprob_out, d_row_max_lse, d_status, stream):
    _call("dash_sample", d_logits, ld, n_rows, vocab, d_row_of, d_seq_uid, d_step, C.c_float(temperature),
          C.c_uint64(seed), d_tokens_out, d_logprob_out, d_row_max_lse, d_status, stream)


def dash_group_advantage_filter(d_rewards, n_groups, group, mode, eps, tau, d_adv, d_kept_idx, d_kept_count, stream):
    _call("dash_group_advantage_filter", d_rewards, n_groups, group, mode, C.c_float(eps), C.c_float(tau), d_adv,
          d_kept_idx, d_kept_count, stream)


def dash_live_compact(d_tok, d_slot, d_pos, d_step, d_uid, d_budget, eos_id, n_rows, d_tok_out, d_slot_out,
                      d_pos_out, d_step_out, d_uid_out, d_count, stream):
    _call("dash_live_compact", d_tok, d_slot, d_pos, d_step, d_uid, d_budget, eos_id, n_rows, d_tok_out, d_slot_out,
          d_pos_out, d_step_out, d_uid_out, d_count, stream)


def dash_rollout_workspace_bytes(model, n_prompts, prompt_len, group, max_ctx) -> int:
    return load().dash_rollout_workspace_bytes(model, n_prompts, prompt_len, group, max_ctx)


def dash_rollout(model, kv, d_prompts, n_prompts, prompt_len, group, gen_len, budgets, temperature, seed,
                 d_out_tokens, d_out_logprobs, use_graph, d_ws, ws_bytes, stream):
    b = i32_array(budgets) if budgets is not None else None
    _call("dash_rollout", model, kv, d_prompts, n_prompts, prompt_len, group, gen_len, b, C.c_float(temperature),
          C.c_uint64(seed), d_out_tokens, d_out_logprobs, int(use_graph), d_ws, ws_bytes, stream)


def dash_bf16_round_check() -> int:
    """Number of float32 inputs on which the kernels' bf16 conversion differs from integer rounding."""
    n = C.c_uint64()
    _call("dash_bf16_round_check", C.byref(n))
    return n.value


def dash_sampler_check() -> tuple[float, float]:
    """(largest |cheap - exact| Gumbel noise over all inputs, the sampler's screening tolerance)."""
    err, tol = C.c_double(), C.c_double()
    _call("dash_sampler_check", C.byref(err), C.byref(tol))
    return err.value, tol.value


def dash_teacher_forced_workspace_bytes(model: int, seqs_per_chunk: int, seq_len: int, prompt_len: int) -> int:
    return load().dash_teacher_forced_workspace_bytes(model, seqs_per_chunk, seq_len, prompt_len)


def dash_teacher_forced_logprobs(model: int, kv: int, d_tokens: int, n_seqs: int, seq_len: int, prompt_len: int,
                                 d_logprobs: int, d_ws: int, ws_bytes: int, stream: int | None) -> None:
    _call("dash_teacher_forced_logprobs", model, kv, d_tokens, n_seqs, seq_len, prompt_len, d_logprobs, d_ws,
          ws_bytes, stream)


def dash_pg_loss(d_logprobs: int, ld: int, T: int, d_lengths: int | None, d_adv: int, d_kept: int, d_kept_count: int,
                 n_total: int, d_loss: int, d_seq_logprob: int | None, stream: int | None) -> None:
    _call("dash_pg_loss", d_logprobs, ld, T, d_lengths, d_adv, d_kept, d_kept_count, n_total, d_loss, d_seq_logprob,
          stream)


def dash_policy_loss(d_logprobs: int, d_logprobs_old: int | None, d_kl: int | None, ld: int, T: int,
                     d_lengths: int | None, d_adv: int, d_kept: int, d_kept_count: int, n_total: int,
                     clip_eps: float, beta: float, d_loss: int, d_stats: int | None, stream: int | None) -> None:
    _call("dash_policy_loss", d_logprobs, d_logprobs_old, d_kl, ld, T, d_lengths, d_adv, d_kept, d_kept_count,
          n_total, C.c_double(clip_eps), C.c_double(beta), d_loss, d_stats, stream)


def dash_logits_kl(d_theta: int, d_base: int, ld: int, rows: int, vocab: int, d_kl: int, d_kl_rev: int | None,
                   stream: int | None) -> None:
    _call("dash_logits_kl", d_theta, d_base, ld, rows, vocab, d_kl, d_kl_rev, stream)


def dash_teacher_forced_kl_workspace_bytes(model: int, seqs_per_chunk: int, seq_len: int, prompt_len: int) -> int:
    return load().dash_teacher_forced_kl_workspace_bytes(model, seqs_per_chunk, seq_len, prompt_len)


def dash_teacher_forced_kl(model: int, base: int, kv: int, d_tokens: int, n_seqs: int, seq_len: int, prompt_len: int,
                           d_logprobs: int | None, d_kl: int, d_kl_rev: int | None, d_ws: int, ws_bytes: int,
                           stream: int | None) -> None:
    _call("dash_teacher_forced_kl", model, base, kv, d_tokens, n_seqs, seq_len, prompt_len, d_logprobs, d_kl,
          d_kl_rev, d_ws, ws_bytes, stream)


def dash_profile_enable(class_mask: int) -> None:
    _call("dash_profile_enable", class_mask)


def dash_profile_layer(layer: int) -> None:
    _call("dash_profile_layer", layer)


def dash_profile_read(reset: bool = True) -> dict:
    """{class name: (milliseconds, launches)} of the timed launches."""
    n = len(K_CLASSES)
    ms = (C.c_double * n)()
    cnt = (C.c_int64 * n)()
    _call("dash_profile_read", ms, cnt, int(reset))
    return {K_CLASSES[i]: (ms[i], cnt[i]) for i in range(n)}
