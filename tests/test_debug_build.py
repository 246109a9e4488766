"""The debug build, liblora_mi355x_debug.so (CPU only).

It exports the release library's ABI, says it is the debug build, and refuses
an op whose outputs overlap its inputs or each other (X / Y, the workspace,
the id array, the table's adapter weights) with LORA_ERR_ALIAS before it
enqueues anything.  Every call here returns before any HIP call: the pointers
are fake, 16-byte aligned and never dereferenced on the host."""
import ctypes
import os

import pytest

from paper_2601_07376_amd import lora
from test_abi import declared_functions

pytestmark = pytest.mark.skipif(
    not (os.path.exists(lora.LIB_PATH) and os.path.exists(lora.DEBUG_LIB_PATH)),
    reason="liblora_mi355x.so / liblora_mi355x_debug.so not built")

ALIAS = 11
BASE = 0x1000000        # fake device addresses, far apart unless a case overlaps them


@pytest.fixture
def D():
    return lora.lib(debug=True)


def test_both_libraries_export_the_abi(D):
    names = declared_functions()
    for L in (lora.lib(), D):
        for name in names:
            assert hasattr(L, name), f"{name} not exported"


def test_build_flags(D):
    assert lora.lib().lora_build_flags() == 0
    assert D.lora_build_flags() == lora.LORA_BUILD_DEBUG


def test_plan_poke_is_debug_only(D):
    # the release library refuses before looking at its arguments
    assert lora.lib().lora_debug_plan_poke(None, lora.LORA_PLAN_PERM, 0, 0, None) == 10
    assert b"debug build" in lora.lib().lora_last_error()
    assert D.lora_debug_plan_poke(None, lora.LORA_PLAN_PERM, 0, 0, None) == 1


class IdsCall:
    """lora_apply_ids on the debug library with fake buffers: X bf16 [n, 1024],
    Y f32 [n, 512], ids int32 [n], the workspace, slot 1's A [16, 1024] and
    B [512, 16] (bf16); each placed at its own offset from BASE."""

    def __init__(self, D, n=100):
        self.D, self.n = D, n
        self.h = ctypes.c_void_p()
        meta = ctypes.c_void_p(BASE)
        assert D.lora_table_create(4, 1024, 512, lora.LORA_BF16, meta, D.lora_table_device_bytes(4),
                                   ctypes.byref(self.h)) == 0
        self.pos = dict(X=BASE + 0x100000, Y=BASE + 0x200000, idx=BASE + 0x300000,
                        ws=BASE + 0x400000, A=BASE + 0x500000, B=BASE + 0x600000)
        self.size = dict(X=n * 1024 * 2, Y=n * 512 * 4, idx=n * 4, A=16 * 1024 * 2, B=512 * 16 * 2)

    def __call__(self, **moved):
        p = dict(self.pos, **moved)
        D = self.D
        assert D.lora_table_set(self.h, 1, 16, 1.0, ctypes.c_void_p(p["A"]), ctypes.c_void_p(p["B"])) == 0
        need = D.lora_apply_ids_workspace_bytes(self.h, self.n)
        v = lambda k: ctypes.c_void_p(p[k])
        st = D.lora_apply_ids(self.h, self.n, v("idx"), v("X"), lora.LORA_BF16, 1024, v("Y"),
                              lora.LORA_F32, 512, v("ws"), need, None)
        return st, D.lora_last_error().decode()

    def close(self):
        self.D.lora_table_destroy(self.h)


@pytest.mark.parametrize("moved,names", [
    (dict(Y=BASE + 0x100000 + 4096), ("Y", "X")),                      # Y inside X
    (dict(Y=BASE + 0x100000 + 100 * 2048 - 16), ("Y", "X")),           # Y's first bytes on X's last
    (dict(ws=BASE + 0x200000 + 512), ("the workspace", "Y")),          # workspace inside Y
    (dict(A=BASE + 0x200000 + 1024), ("Y", "A of slot 1")),            # Y over slot 1's A
    (dict(B=BASE + 0x400000), ("the workspace", "B of slot 1")),       # workspace over B
    (dict(idx=BASE + 0x400000 + 64), ("the workspace", "idx")),        # ids inside the workspace
    (dict(Y=BASE + 64), ("Y", "the slot table")),                      # Y over the slot table
])
def test_apply_ids_overlaps_are_refused(D, moved, names):
    call = IdsCall(D)
    st, msg = call(**moved)
    call.close()
    assert st == ALIAS, msg
    assert "lora_apply_ids" in msg
    for nm in names:
        assert nm in msg, msg


def test_adjacent_buffers_do_not_overlap(D):
    """Y starting exactly where X ends is no overlap: the only one reported is
    the planted workspace / ids one."""
    call = IdsCall(D)
    x_end = call.pos["X"] + call.size["X"]
    st, msg = call(Y=x_end, idx=BASE + 0x400000)
    call.close()
    assert st == ALIAS
    assert "Y overlaps" not in msg and "overlaps Y" not in msg, msg
    assert "idx" in msg
