"""C-ABI checks that need no GPU: the library loads, exports every entry point
include/bp.h declares, and rejects bad arguments before any device work."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bp.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(bp_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def bp():
    from paper_1801_01554_amd import bp as mod
    mod.lib()
    return mod


def test_header_declares_the_binding_names(bp):
    assert _declared() == sorted(bp.EXPORTS)


def test_library_exports_every_declared_symbol(bp):
    L = bp.lib()
    for name in _declared():
        assert hasattr(L, name), name


def test_create_rejects_bad_sizes_before_device_work(bp):
    for sizes in ([], [5], [5, 0], [3, -1, 2]):
        rc, h = bp.bp_create(sizes)
        assert rc == bp.BP_EINVAL and not h.value
        assert "bp_create" in bp.bp_last_error(None)
    h = ctypes.c_void_p()
    assert bp.lib().bp_create(None, 3, ctypes.byref(h)) == bp.BP_EINVAL
    arr = (ctypes.c_int32 * 2)(4, 2)
    assert bp.lib().bp_create(arr, 2, None) == bp.BP_EINVAL


def test_null_net_is_rejected(bp):
    L = bp.lib()
    assert L.bp_num_weights(None) == -1
    assert L.bp_set_weights(None, None, 0) == bp.BP_EINVAL
    assert L.bp_get_weights(None, None, 0) == bp.BP_EINVAL
    assert L.bp_set_momentum(None, None, 0) == bp.BP_EINVAL
    assert L.bp_get_momentum(None, None, 0) == bp.BP_EINVAL
    assert L.bp_set_stream(None, None) == bp.BP_EINVAL
    assert L.bp_train_batches(None, None, None, 0, 1, 0.1, 0.9, None) == bp.BP_EINVAL
    assert L.bp_train_batches_onehot(None, None, 7, None, 0, 1, 0.1, 0.9, None) == bp.BP_EINVAL
    assert L.bp_forward(None, None, 0, None) == bp.BP_EINVAL
    assert L.bp_forward_onehot(None, None, 7, 0, None) == bp.BP_EINVAL
    assert L.bp_set_context(None, 0, None, None) == bp.BP_EINVAL
    assert L.bp_train_sequences(None, None, None, None, None, 0, 1, 1, 0.1, 0.9, None) == bp.BP_EINVAL
    assert L.bp_forward_sequences(None, None, None, 0, 1, None) == bp.BP_EINVAL
    assert L.bp_set_sigmoid(None, 1) == bp.BP_EINVAL
    assert L.bp_set_fault_limit(None, 1.0) == bp.BP_EINVAL
    assert L.bp_get_fault_count(None, None) == bp.BP_EINVAL
    assert L.bp_checkpoint_save(None) == bp.BP_EINVAL
    assert L.bp_checkpoint_restore(None) == bp.BP_EINVAL
    assert L.bp_guard_config(None, 1, 2.0) == bp.BP_EINVAL
    assert L.bp_guard_epoch(None, 1.0, None) == bp.BP_EINVAL
    assert L.bp_profile(None, 1) == bp.BP_EINVAL
    assert L.bp_set_graph_replay(None, 1) == bp.BP_EINVAL
    L.bp_destroy(None)   # no-op
