"""The C-ABI library loads, exports every function include/smallkv.h declares,
and rejects host-detectable misuse before touching the GPU (no compute calls
here: this file runs without a GPU)."""
import ctypes as C
import os
import re

import pytest

from paper_2508_02751_amd import smallkv as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "smallkv.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(smallkv_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_four_stage_calls():
    names = declared_functions()
    for f in ("smallkv_small_attn", "smallkv_partition", "smallkv_hybrid_attn", "smallkv_step"):
        assert f in names


def test_library_exports_every_declared_symbol():
    L = S.lib()
    for name in declared_functions():
        assert hasattr(L, name), name
    assert set(S.EXPORTS) >= set(declared_functions())


def test_abi_version_and_status_strings():
    L = S.lib()
    assert L.smallkv_abi_version() == 8
    assert L.smallkv_status_string(0) == b"ok"
    assert L.smallkv_status_string(-3) == b"workspace too small"
    assert L.smallkv_status_string(123) == b"unknown status"


def _fake_step(**over):
    """A descriptor with plausible (never dereferenced) pointers."""
    p = 0x1000
    b = S.Batch(batch=1, n_cap=512, seq_len=p, k_crit=p, k_marg=p, k_recent=None, kc_cap=64,
                km_cap=128)
    sm = S.Model(1, 14, 2, 64, S.BF16, 0.125, p, p, p, 512, None, None, p)
    lg = S.Model(1, 28, 4, 128, S.BF16, 0.088, p, p, p, 512, None, None, p)
    st = S.Step(b, sm, lg, p, 0, p, p, p, p, p, p, p, S.SELECT_HEAD, None)
    for k, v in over.items():
        obj, field = k.split("__")
        setattr({"b": st.batch, "s": st.small, "l": st.large, "st": st}[obj], field, v)
    return st


@pytest.mark.parametrize("over,status", [
    ({"s__head_dim": 96}, S.EUNSUPPORTED),
    ({"s__n_q_heads": 13}, S.EINVAL),
    ({"s__dtype": 7}, S.EINVAL),
    ({"s__q": None}, S.EINVAL),
    ({"b__batch": 0}, S.EINVAL),
    ({"b__kc_cap": 0}, S.EINVAL),
    ({"b__seq_len": None}, S.EINVAL),
    ({"s__n_rows": 100}, S.EINVAL),
    ({"s__k_slot": 0x1000}, S.EINVAL),
    ({"s__n_q_heads": 34, "s__n_kv_heads": 2}, S.EUNSUPPORTED),
    ({"s__held": 0x1000}, S.EINVAL),                      # held rows without positions
    ({"s__row_pos": 0x1000}, S.EINVAL),                   # positions without held rows
    ({"s__held": 0x1000, "s__row_pos": 0x1000, "s__n_rows": 600}, S.EINVAL),  # > n_cap
    ({"l__held": 0x1000, "l__row_pos": 0x1000}, S.EINVAL),  # small model only
    ({"st__select": 3}, S.EINVAL),
])
def test_workspace_size_rejects_bad_small_model(over, status):
    n = C.c_size_t()
    assert S.lib().smallkv_workspace_size(C.byref(_fake_step(**over)), C.byref(n)) == status


@pytest.mark.parametrize("over,status", [
    ({"l__head_dim": 80}, S.EUNSUPPORTED),
    ({"l__n_kv_heads": 3}, S.EINVAL),
    ({"st__mode": 9}, S.EINVAL),
    ({"st__head_map": None}, S.EINVAL),
    ({"st__logits": None}, S.EINVAL),
    ({"l__k_slot": 0x1000}, S.EINVAL),          # one slot map without the other
    ({"l__n_rows": 100}, S.EINVAL),             # compact rows need slot maps
    ({"b__kc_cap": 20000, "l__dtype": S.F32}, S.EUNSUPPORTED),  # per-head kernel's LDS
    ({"st__select": 2}, S.EINVAL),               # accumulated scores without their state
    ({"st__select": 2, "st__acc_score": 0x1000, "s__held": 0x1000, "s__row_pos": 0x1000,
      "s__n_rows": 200}, S.EUNSUPPORTED),        # ... or over a compressed small cache
])
def test_step_rejects_before_launch(over, status):
    st = _fake_step(**over)
    assert S.lib().smallkv_step(C.byref(st), None, 0, None) == status


def test_step_needs_workspace():
    st = _fake_step()
    n = C.c_size_t()
    assert S.lib().smallkv_workspace_size(C.byref(st), C.byref(n)) == 0 and n.value > 0
    assert S.lib().smallkv_step(C.byref(st), None, 0, None) == S.EWORKSPACE
    assert S.lib().smallkv_step(C.byref(st), C.c_void_p(0x1000), n.value - 1, None) == S.EWORKSPACE


def test_partition_and_hybrid_reject_nulls():
    b = S.Batch(batch=1, n_cap=512, seq_len=0x1000, k_crit=0x1000, k_marg=0x1000, k_recent=None,
                kc_cap=64, km_cap=128)
    L = S.lib()
    assert L.smallkv_partition(C.byref(b), None, 14, None, 1, 1, 1, 1, 1, 1, None, 0,
                               None) == S.EINVAL
    lg = S.Model(1, 28, 4, 128, S.BF16, 0.088, 1, 1, 1, 512, None, None, 1)
    assert L.smallkv_hybrid_attn(C.byref(b), C.byref(lg), None, 14, 1, 1, 1, 1, 0, 0, None, 0,
                                 None) == S.EINVAL


def _fake_match(**over):
    """A matching descriptor with plausible (never dereferenced) 16-byte aligned pointers."""
    p = 0x1000
    lg = S.Window(28, 28, 4, 128, S.BF16, 0.088, p, p)
    sm = S.Window(24, 14, 2, 64, S.BF16, 0.125, p, p)
    m = S.Match(1, 200, p, p, lg, sm, p, None, None)
    for k, v in over.items():
        obj, field = k.split("__")
        setattr({"m": m, "l": m.large, "s": m.small}[obj], field, v)
    return m


def test_header_declares_the_matching_calls():
    names = declared_functions()
    assert "smallkv_match" in names and "smallkv_match_workspace_size" in names


@pytest.mark.parametrize("over,status", [
    ({"m__w_cap": 0}, S.EINVAL),
    ({"m__w_cap": 257}, S.EUNSUPPORTED),
    ({"m__batch": 0}, S.EINVAL),
    ({"m__win_len": None}, S.EINVAL),
    ({"m__top_k": None}, S.EINVAL),
    ({"m__head_map": None}, S.EINVAL),
    ({"l__head_dim": 96}, S.EUNSUPPORTED),
    ({"s__n_kv_heads": 3}, S.EINVAL),
    ({"s__dtype": 5}, S.EINVAL),
    ({"l__q": 0x1004}, S.EINVAL),               # not 16-byte aligned
    ({"s__k": None}, S.EINVAL),
    ({"l__n_layers": 3000}, S.EUNSUPPORTED),    # more heads than one grid dimension
])
def test_match_rejects_before_launch(over, status):
    m = _fake_match(**over)
    n = C.c_size_t()
    assert S.lib().smallkv_match_workspace_size(C.byref(m), C.byref(n)) == status
    assert S.lib().smallkv_match(C.byref(m), C.c_void_p(0x1000), 1 << 40, None) == status


def test_match_workspace_size_and_check():
    m = _fake_match()
    n = C.c_size_t()
    assert S.lib().smallkv_match_workspace_size(C.byref(m), C.byref(n)) == 0
    H = 28 * 28 + 24 * 14
    assert n.value >= H * 200 * 200 * 4 + H * 200 * 8 + H * 4 * 8  # S, row (max, sum), bitsets
    assert S.lib().smallkv_match(C.byref(m), None, 0, None) == S.EWORKSPACE
    assert S.lib().smallkv_match(C.byref(m), C.c_void_p(0x1000), n.value - 1, None) == S.EWORKSPACE


def test_small_model_held_rows_accepted():
    st = _fake_step(s__held=0x1000, s__row_pos=0x1000, s__n_rows=200)
    n = C.c_size_t()
    assert S.lib().smallkv_workspace_size(C.byref(st), C.byref(n)) == 0 and n.value > 0


def test_partition_with_held_rows_checks_the_small_model():
    b = S.Batch(batch=1, n_cap=512, seq_len=0x1000, k_crit=0x1000, k_marg=0x1000, k_recent=None,
                kc_cap=64, km_cap=128)
    sm = S.Model(1, 14, 2, 64, S.BF16, 0.125, 0x1000, 0x1000, 0x1000, 200, None, None, 0x1000,
                 0x1000, 0x1000)
    L = S.lib()
    # 13 heads for a 14-head small model
    assert L.smallkv_partition(C.byref(b), C.byref(sm), 13, 1, 1, 1, 1, 1, 1, 1, None, 0,
                               None) == S.EINVAL
    sm.row_pos = None  # held rows without positions
    assert L.smallkv_partition(C.byref(b), C.byref(sm), 14, 1, 1, 1, 1, 1, 1, 1, None, 0,
                               None) == S.EINVAL


def test_group_selection_limits():
    # a compressed small cache, or more than 16 query heads per kv head
    for over in ({"s__held": 0x1000, "s__row_pos": 0x1000, "s__n_rows": 200},
                 {"l__n_q_heads": 32, "l__n_kv_heads": 1}):
        st = _fake_step(st__select=S.SELECT_GROUP, **over)
        assert S.lib().smallkv_step(C.byref(st), C.c_void_p(0x1000), 1 << 40, None) == S.EUNSUPPORTED
    st = _fake_step(st__select=S.SELECT_GROUP)
    n = C.c_size_t()
    assert S.lib().smallkv_workspace_size(C.byref(st), C.byref(n)) == 0 and n.value > 0


def _fake_store(**over):
    """A well-formed retained-store descriptor over fake 16-byte aligned
    addresses (Qwen2-7B shapes, batch 2, N 8192); `over` replaces fields."""
    b = S.Batch(batch=2, n_cap=8192, seq_len=0x1000, k_crit=0x1000, k_marg=0x1000, k_recent=None,
                kc_cap=820, km_cap=1640)
    st = S.Store(b, 28, 28, 4, 128, S.BF16, 0x1000, 336, S.SELECT_HEAD, 0x1000, 0x1000, 0x2000,
                 0x3000, 4096, None, None, None, None, 0x4000, 0x5000, 0x6000, 0x7000, None)
    for k, v in over.items():
        if k.startswith("b__"):
            setattr(st.batch, k[3:], v)
        else:
            setattr(st, k, v)
    return st


def test_header_declares_the_store_calls():
    names = declared_functions()
    assert "smallkv_store_update" in names and "smallkv_store_workspace_size" in names


def test_store_workspace_size():
    st = _fake_store()
    n = C.c_size_t()
    assert S.lib().smallkv_store_workspace_size(C.byref(st), C.byref(n)) == 0
    units = 2 * 28 * 4
    assert n.value == 2 * units * 4096 * 4 + 2 * units * 4  # both unions' row sources, sizes
    assert S.lib().smallkv_store_workspace_size(C.byref(st), None) == S.EINVAL
    # workspace checks come before any device call
    assert S.lib().smallkv_store_update(C.byref(st), None, 0, None) == S.EWORKSPACE
    assert S.lib().smallkv_store_update(C.byref(st), C.c_void_p(0x1000), n.value - 1,
                                        None) == S.EWORKSPACE


@pytest.mark.parametrize("over,status", [
    ({"b__n_cap": 131073}, S.EUNSUPPORTED),   # past the index kernel's LDS bitmaps
    ({"head_dim": 96}, S.EUNSUPPORTED),
    ({"rows": 0}, S.EINVAL),
    ({"n_q_heads": 30}, S.EINVAL),            # not a multiple of the kv heads
    ({"dtype": 7}, S.EINVAL),
    ({"select": 9}, S.EINVAL),
    ({"head_map": None}, S.EINVAL),
    ({"crit_idx": None}, S.EINVAL),
    ({"marg_idx": None}, S.EINVAL),           # km_cap > 0 needs the marginal lists
    ({"full_k": 0x2004}, S.EINVAL),           # not 16-byte aligned
    ({"new_v": None}, S.EINVAL),
    ({"k_slot": None}, S.EINVAL),
    ({"old_k": 0x8000}, S.EINVAL),            # part of an old store only
    ({"old_k": 0x4000, "old_v": 0x8000, "old_k_slot": 0x9000, "old_v_slot": 0xa000},
     S.EINVAL),                               # the old store is the new one
    ({"b__batch": 0}, S.EINVAL),
])
def test_store_rejects_before_launch(over, status):
    st = _fake_store(**over)
    n = C.c_size_t()
    assert S.lib().smallkv_store_workspace_size(C.byref(st), C.byref(n)) == status
    assert S.lib().smallkv_store_update(C.byref(st), C.c_void_p(0x1000), 1 << 40, None) == status


def test_store_accepts_a_whole_old_store():
    st = _fake_store(old_k=0x8000, old_v=0x9000, old_k_slot=0xa000, old_v_slot=0xb000)
    n = C.c_size_t()
    assert S.lib().smallkv_store_workspace_size(C.byref(st), C.byref(n)) == 0


def test_noalloc_step_checks_before_touching_a_device():
    """smallkv_step_noalloc validates like smallkv_step and refuses a step
    whose workspace exceeds its static scratch, before any device call."""
    L = S.lib()
    assert L.smallkv_step_noalloc(None, None) == S.EINVAL
    assert L.smallkv_step_noalloc(C.byref(_fake_step(**{"st__mode": 9})), None) == S.EINVAL
    # one selection per kv group over 16 x 32768 tokens: ~590 MB of workspace
    big = _fake_step(**{"b__batch": 16, "b__n_cap": 32768, "b__kc_cap": 1638, "b__km_cap": 4915,
                        "s__n_layers": 16, "s__n_q_heads": 32, "s__n_kv_heads": 8,
                        "s__n_rows": 32768, "l__n_layers": 32, "l__n_q_heads": 32,
                        "l__n_kv_heads": 8, "l__n_rows": 32768, "st__select": S.SELECT_GROUP})
    n = C.c_size_t()
    assert L.smallkv_workspace_size(C.byref(big), C.byref(n)) == 0
    assert n.value > S.NOALLOC_SCRATCH_BYTES
    assert L.smallkv_step_noalloc(C.byref(big), None) == S.EWORKSPACE
    # the header's limit and the binding's agree
    text = open(os.path.join(ROOT, "include", "smallkv.h")).read()
    assert "#define SMALLKV_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)" in text
    assert S.NOALLOC_SCRATCH_BYTES == 32 << 20



def test_layer_range_and_its_workspace_checked_on_the_host():
    L = S.lib()
    b = S.Batch(batch=2, n_cap=512, seq_len=0x1000, k_crit=0x1000, k_marg=0x1000, k_recent=None,
                kc_cap=64, km_cap=128)
    lg = S.Model(4, 28, 4, 128, S.BF16, 0.088, 1, 1, 1, 512, None, None, 1)
    n = C.c_size_t()
    assert L.smallkv_hybrid_attn_workspace_size(C.byref(b), C.byref(lg), 1, 14, C.byref(n)) == 0
    one = n.value
    assert L.smallkv_hybrid_attn_workspace_size(C.byref(b), C.byref(lg), 4, 14, C.byref(n)) == 0
    assert one > 0 and n.value > 0
    for bad in (0, 5):
        assert L.smallkv_hybrid_attn_workspace_size(C.byref(b), C.byref(lg), bad, 14,
                                                    C.byref(n)) == S.EINVAL
    for l0, cnt in ((-1, 1), (3, 2), (0, 0), (4, 1)):
        assert L.smallkv_hybrid_attn_layers(C.byref(b), C.byref(lg), l0, cnt, 1, 14, 1, 1, 1, 1,
                                            0, 0, C.c_void_p(0x1000), 1 << 30, None) == S.EINVAL
    # a workspace below the layer call's own size
    assert L.smallkv_hybrid_attn_layers(C.byref(b), C.byref(lg), 0, 1, 1, 14, 1, 1, 1, 1, 0, 0,
                                        C.c_void_p(0x1000), one - 1, None) == S.EWORKSPACE
