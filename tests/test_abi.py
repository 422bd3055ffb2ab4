"""Host-side checks of the C ABI: every declared entry point is exported,
the binding mirrors the header, and argument validation that runs before any
HIP call returns the documented status codes (no GPU needed)."""
import ctypes
import os
import re

import pytest

from paper_2602_01762_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "prism_draft.h")

needs_lib = pytest.mark.skipif(not os.path.exists(B.LIB_PATH), reason="library not built")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(prism_\w+)\s*\(", src)))


def test_header_declares_north_star_calls():
    fns = declared_functions()
    for name in ("prism_draft_load_params", "prism_draft_step", "prism_draft_chain",
                 "prism_draft_tree"):
        assert name in fns


def test_binding_mirrors_header():
    assert sorted(B.EXPORTS) == declared_functions()


@needs_lib
def test_library_exports_every_declared_symbol():
    L = ctypes.CDLL(B.LIB_PATH)
    for name in declared_functions():
        assert hasattr(L, name), name


def _struct_sizes_from_header():
    return {"prism_config": 17 * 4, "prism_param_set": 10 * 8 + 8,
            "prism_batch": 8 + 6 * 8 + 8}


def test_struct_layouts():
    s = _struct_sizes_from_header()
    assert ctypes.sizeof(B.prism_config) == s["prism_config"]
    assert ctypes.sizeof(B.prism_param_set) == s["prism_param_set"]
    assert ctypes.sizeof(B.prism_batch) == s["prism_batch"]


def _cfg(**kw):
    c = B.prism_config(hidden=256, n_q_heads=4, n_kv_heads=4, head_dim=64, ffn=688, vocab=4096,
                       n_sets=3, max_steps=3, feat_width=256, rope_theta=1e4, rms_eps=1e-5,
                       dtype=B.PRISM_F32, kv_block_size=16, max_batch=1, max_blocks_per_seq=9,
                       tree_width=0, tree_nodes=0)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


@needs_lib
@pytest.mark.parametrize("bad,code", [
    (dict(dtype=7), -1),
    (dict(hidden=0), -1),
    (dict(n_kv_heads=3), -2),            # 4 % 3 != 0
    (dict(n_q_heads=36, n_kv_heads=4), -2),   # 9 query heads per KV head
    (dict(hidden=250), -2),              # not a multiple of 16 (fp32 tiling)
    (dict(vocab=4097), -2),
    (dict(head_dim=66), -2),
    (dict(max_steps=64), -2),
    (dict(max_batch=65), -2),            # more than 64 rows per pass
    (dict(tree_width=8, tree_nodes=0, max_steps=3), -2),
    (dict(tree_width=8, tree_nodes=60, max_steps=9, max_batch=1), -2),  # > 64 draft slots
])
def test_create_rejects_bad_config(bad, code):
    L = B.lib()
    h = ctypes.c_void_p()
    st = L.prism_create(ctypes.byref(_cfg(**bad)), ctypes.byref(h))
    assert st == code
    assert h.value is None
    assert L.prism_last_error(None)


@needs_lib
def test_create_null_args():
    L = B.lib()
    assert L.prism_create(None, None) == -1
    h = ctypes.c_void_p()
    assert L.prism_create(None, ctypes.byref(h)) == -1
    assert L.prism_draft_chain(None, None, 1, None, None, None, None) == -1
    assert L.prism_draft_tree(None, None, 1, None, None) == -1
    assert L.prism_draft_step(None, 1, None, None) == -1
