"""ctypes binding of libprism_draft.so (include/prism_draft.h).

Argument marshalling only: every step of the drafting path runs in the HIP
library.  Device buffers are torch tensors (their data pointers are passed);
the stream is torch's current HIP stream unless one is given.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libprism_draft.so")

PRISM_F32, PRISM_BF16 = 0, 1
STATUS = {0: "PRISM_OK", -1: "PRISM_ERR_INVALID_ARG", -2: "PRISM_ERR_SHAPE",
          -3: "PRISM_ERR_NOT_LOADED", -4: "PRISM_ERR_UNSUPPORTED",
          -5: "PRISM_ERR_OUT_OF_MEMORY", -6: "PRISM_ERR_HIP", -7: "PRISM_ERR_CAPACITY",
          -8: "PRISM_ERR_NONFINITE"}
EXPORTS = ("prism_create", "prism_destroy", "prism_last_error", "prism_draft_load_shared",
           "prism_draft_load_params", "prism_set_step_map", "prism_draft_step",
           "prism_draft_chain", "prism_draft_chain_catchup", "prism_draft_chain_sample",
           "prism_draft_tree", "prism_score_tree", "prism_verify_chain",
           "prism_verify_chain_static",
           "prism_verify_tree",
           "prism_device_status",
           "prism_profile_enable", "prism_profile_read", "prism_profile_pairs",
           "prism_graph_cache")

c_i32, c_u64, c_f32, c_vp = ctypes.c_int32, ctypes.c_uint64, ctypes.c_float, ctypes.c_void_p


class prism_config(ctypes.Structure):
    _fields_ = [("hidden", c_i32), ("n_q_heads", c_i32), ("n_kv_heads", c_i32),
                ("head_dim", c_i32), ("ffn", c_i32), ("vocab", c_i32), ("n_sets", c_i32),
                ("max_steps", c_i32), ("feat_width", c_i32), ("rope_theta", c_f32),
                ("rms_eps", c_f32), ("dtype", c_i32), ("kv_block_size", c_i32),
                ("max_batch", c_i32), ("max_blocks_per_seq", c_i32), ("tree_width", c_i32),
                ("tree_nodes", c_i32), ("max_new_rows", c_i32)]


class prism_param_set(ctypes.Structure):
    _fields_ = [("d_w_fc", c_vp), ("d_g1", c_vp), ("d_w_q", c_vp), ("d_w_k", c_vp),
                ("d_w_v", c_vp), ("d_w_o", c_vp), ("d_g2", c_vp), ("d_w_gate", c_vp),
                ("d_w_up", c_vp), ("d_w_down", c_vp), ("feat_width", c_i32)]


class prism_batch(ctypes.Structure):
    _fields_ = [("batch", c_i32), ("d_tokens", c_vp), ("d_features", c_vp),
                ("d_ctx_lens", c_vp), ("d_k_pool", c_vp), ("d_v_pool", c_vp),
                ("d_block_table", c_vp), ("n_pool_blocks", c_i32)]


class prism_catchup(ctypes.Structure):
    _fields_ = [("total_rows", c_i32), ("d_offsets", c_vp), ("d_tokens", c_vp),
                ("d_features", c_vp)]


class prism_step_io(ctypes.Structure):
    _fields_ = [("rows", c_i32), ("d_tokens", c_vp), ("d_feat", c_vp), ("feat_dtype", c_i32),
                ("d_feat_rows", c_vp), ("d_seq", c_vp), ("d_pos", c_vp), ("d_slot", c_vp),
                ("d_tree_bits", c_vp), ("kv", ctypes.POINTER(prism_batch)), ("topk", c_i32),
                ("d_hidden_out", c_vp), ("d_topk_ids", c_vp), ("d_topk_logp", c_vp),
                ("d_logits", c_vp)]


class prism_tree_out(ctypes.Structure):
    _fields_ = [("d_tokens", c_vp), ("d_parent", c_vp), ("d_depth", c_vp), ("d_score", c_vp),
                ("d_mask", c_vp), ("d_cand_tokens", c_vp), ("d_cand_parent", c_vp),
                ("d_cand_score", c_vp), ("d_frontier", c_vp), ("d_logits", c_vp)]


class PrismError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("%s: %s" % (STATUS.get(status, status), msg))
        self.status = status


_lib = None


def lib():
    """Load the HIP library; fails loudly if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libprism_draft.so is not built (run __graft_entry__.build()): "
                              + LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER
        L.prism_create.argtypes = [P(prism_config), P(c_vp)]
        L.prism_destroy.argtypes = [c_vp]
        L.prism_destroy.restype = None
        L.prism_last_error.argtypes = [c_vp]
        L.prism_last_error.restype = ctypes.c_char_p
        L.prism_draft_load_shared.argtypes = [c_vp, c_vp, c_vp, c_vp, c_vp]
        L.prism_draft_load_params.argtypes = [c_vp, c_i32, P(prism_param_set), c_vp]
        L.prism_set_step_map.argtypes = [c_vp, P(c_i32), c_i32]
        L.prism_draft_step.argtypes = [c_vp, c_i32, P(prism_step_io), c_vp]
        L.prism_draft_chain.argtypes = [c_vp, P(prism_batch), c_i32, c_vp, c_vp, c_vp, c_vp]
        L.prism_draft_chain_catchup.argtypes = [c_vp, P(prism_batch), P(prism_catchup), c_i32,
                                                c_vp, c_vp, c_vp, c_vp]
        L.prism_draft_chain_sample.argtypes = [c_vp, P(prism_batch), c_i32, c_f32, c_vp, c_vp,
                                               c_vp, c_vp, c_vp, c_vp]
        L.prism_draft_tree.argtypes = [c_vp, P(prism_batch), c_i32, P(prism_tree_out), c_vp]
        L.prism_score_tree.argtypes = [c_vp, P(prism_batch), c_i32, c_vp, c_vp, c_vp, c_vp, c_vp]
        L.prism_verify_chain.argtypes = [c_vp, c_i32, c_i32, c_f32, c_vp, c_vp, c_vp, c_vp, c_vp,
                                         c_vp, c_vp]
        L.prism_verify_chain_static.argtypes = [c_i32, c_i32, c_i32, c_f32, c_vp, c_vp, c_vp,
                                                c_vp, c_vp, c_vp, c_vp]
        L.prism_verify_tree.argtypes = [c_vp, c_i32, c_i32, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp,
                                        c_vp]
        L.prism_device_status.argtypes = [c_vp, c_vp]
        L.prism_profile_enable.argtypes = [c_vp, c_i32]
        L.prism_profile_read.argtypes = [c_vp, P(c_f32), P(c_i32)]
        L.prism_profile_pairs.argtypes = [c_vp, P(c_f32), c_i32, P(c_i32)]
        L.prism_graph_cache.argtypes = [c_vp, P(c_i32), P(c_i32)]
        for n in EXPORTS:
            if n not in ("prism_destroy", "prism_last_error"):
                getattr(L, n).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(st: int, ctx) -> None:
    if st != 0:
        msg = lib().prism_last_error(ctx)
        raise PrismError(st, msg.decode() if msg else "")


def ptr(t) -> int:
    """Device pointer of a tensor (0 for None)."""
    return 0 if t is None else int(t.data_ptr())


def cur_stream():
    import torch
    return int(torch.cuda.current_stream().cuda_stream)


# thin wrappers with the C names ------------------------------------------------
def prism_create(cfg: prism_config) -> int:
    h = c_vp()
    _check(lib().prism_create(ctypes.byref(cfg), ctypes.byref(h)), None)
    return h.value


def prism_destroy(ctx: int) -> None:
    lib().prism_destroy(ctx)


def prism_last_error(ctx) -> str:
    m = lib().prism_last_error(ctx)
    return m.decode() if m else ""


def prism_draft_load_shared(ctx, embed, lm_head, final_norm, stream=None):
    _check(lib().prism_draft_load_shared(ctx, ptr(embed), ptr(lm_head), ptr(final_norm),
                                         cur_stream() if stream is None else stream), ctx)


def prism_draft_load_params(ctx, set_idx: int, ps: prism_param_set, stream=None):
    _check(lib().prism_draft_load_params(ctx, set_idx, ctypes.byref(ps),
                                         cur_stream() if stream is None else stream), ctx)


def prism_set_step_map(ctx, f_map):
    arr = (c_i32 * len(f_map))(*[int(x) for x in f_map])
    _check(lib().prism_set_step_map(ctx, arr, len(f_map)), ctx)


def prism_draft_step(ctx, k: int, io: prism_step_io, stream=None):
    _check(lib().prism_draft_step(ctx, k, ctypes.byref(io),
                                  cur_stream() if stream is None else stream), ctx)


def prism_draft_chain(ctx, batch: prism_batch, K: int, out_tokens, out_logits=None,
                      out_hidden=None, stream=None):
    _check(lib().prism_draft_chain(ctx, ctypes.byref(batch), K, ptr(out_tokens), ptr(out_logits),
                                   ptr(out_hidden), cur_stream() if stream is None else stream), ctx)


def prism_draft_chain_catchup(ctx, batch: prism_batch, catchup: prism_catchup, K: int,
                              out_tokens, out_logits=None, out_hidden=None, stream=None):
    _check(lib().prism_draft_chain_catchup(ctx, ctypes.byref(batch), ctypes.byref(catchup), K,
                                           ptr(out_tokens), ptr(out_logits), ptr(out_hidden),
                                           cur_stream() if stream is None else stream), ctx)


def prism_draft_chain_sample(ctx, batch: prism_batch, K: int, temperature: float, uniforms,
                             out_tokens, out_logp=None, out_logits=None, out_hidden=None,
                             stream=None):
    _check(lib().prism_draft_chain_sample(ctx, ctypes.byref(batch), K, float(temperature),
                                          ptr(uniforms), ptr(out_tokens), ptr(out_logp),
                                          ptr(out_logits), ptr(out_hidden),
                                          cur_stream() if stream is None else stream), ctx)


def prism_draft_tree(ctx, batch: prism_batch, depth: int, out: prism_tree_out, stream=None):
    _check(lib().prism_draft_tree(ctx, ctypes.byref(batch), depth, ctypes.byref(out),
                                  cur_stream() if stream is None else stream), ctx)


def prism_score_tree(ctx, batch: prism_batch, n_nodes: int, tokens, depth, mask, logits,
                     stream=None):
    _check(lib().prism_score_tree(ctx, ctypes.byref(batch), n_nodes, ptr(tokens), ptr(depth),
                                  ptr(mask), ptr(logits),
                                  cur_stream() if stream is None else stream), ctx)


def prism_verify_chain(ctx, batch: int, K: int, temperature: float, target_logits, draft_logits,
                       draft_tokens, uniforms, n_accepted, next_token, stream=None):
    _check(lib().prism_verify_chain(ctx, batch, K, float(temperature), ptr(target_logits),
                                    ptr(draft_logits), ptr(draft_tokens), ptr(uniforms),
                                    ptr(n_accepted), ptr(next_token),
                                    cur_stream() if stream is None else stream), ctx)


def prism_verify_chain_static(vocab: int, batch: int, K: int, temperature: float, target_logits,
                              draft_logits, draft_tokens, uniforms, n_accepted, next_token,
                              stream=None):
    _check(lib().prism_verify_chain_static(vocab, batch, K, float(temperature),
                                           ptr(target_logits), ptr(draft_logits),
                                           ptr(draft_tokens), ptr(uniforms), ptr(n_accepted),
                                           ptr(next_token),
                                           cur_stream() if stream is None else stream), None)


def prism_verify_tree(ctx, batch: int, n_nodes: int, target_logits, tokens, parent, n_accepted,
                      path, next_token, stream=None):
    _check(lib().prism_verify_tree(ctx, batch, n_nodes, ptr(target_logits), ptr(tokens),
                                   ptr(parent), ptr(n_accepted), ptr(path), ptr(next_token),
                                   cur_stream() if stream is None else stream), ctx)


def prism_device_status(ctx, stream=None) -> int:
    """Returns the status code (does not raise), so tests can inspect it."""
    return lib().prism_device_status(ctx, cur_stream() if stream is None else stream)


PRISM_PROFILE_LMHEAD, PRISM_PROFILE_PRODUCTS, PRISM_PROFILE_PASSES = 1, 2, 4


def prism_profile_enable(ctx, what=PRISM_PROFILE_LMHEAD):
    """what: PRISM_PROFILE_* bits (True = the LM head), 0 / False = off."""
    _check(lib().prism_profile_enable(ctx, int(what)), ctx)


def prism_profile_read(ctx):
    """(summed LM-head milliseconds, launch count) of the last chain/tree call."""
    ms, n = c_f32(), c_i32()
    _check(lib().prism_profile_read(ctx, ctypes.byref(ms), ctypes.byref(n)), ctx)
    return ms.value, n.value


def prism_profile_pairs(ctx, cap: int = 512):
    """Milliseconds of each event pair of the last drafting call, in launch order."""
    arr, n = (c_f32 * cap)(), c_i32()
    _check(lib().prism_profile_pairs(ctx, arr, cap, ctypes.byref(n)), ctx)
    return list(arr[:min(n.value, cap)])


def prism_graph_cache(ctx):
    """(graphs held, capacity) of the context's captured-graph cache."""
    n, cap = c_i32(), c_i32()
    _check(lib().prism_graph_cache(ctx, ctypes.byref(n), ctypes.byref(cap)), ctx)
    return n.value, cap.value
