"""The C ABI library loads, exports every declared symbol, and rejects bad
arguments on the host before touching the GPU (CPU only: no compute calls)."""
import ctypes
import os
import re

import pytest

from paper_2601_07376_amd import lora

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lora.h")

pytestmark = pytest.mark.skipif(not os.path.exists(lora.LIB_PATH),
                                reason="liblora_mi355x.so not built")

FAKE = 0x10000          # 16-byte aligned, never dereferenced on the host
FAKE_ODD = 0x10002      # misaligned


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lora_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported_and_bound():
    L = lora.lib()
    names = declared_functions()
    assert len(names) >= 20
    for name in names:
        assert hasattr(L, name), f"{name} not exported"
        assert name in lora.SIGNATURES, f"{name} has no binding"
    assert set(lora.SIGNATURES) == set(names)


def test_version_and_strings():
    L = lora.lib()
    assert L.lora_abi_version() == 1
    for s in range(12):
        assert L.lora_status_string(s) != b"unknown status"
    assert L.lora_status_string(99) == b"unknown status"


def _create(S=4, d_in=64, d_out=32, w=lora.LORA_BF16, meta=FAKE, nbytes=None):
    L = lora.lib()
    h = ctypes.c_void_p()
    nbytes = L.lora_table_device_bytes(S) if nbytes is None else nbytes
    st = L.lora_table_create(S, d_in, d_out, w, ctypes.c_void_p(meta), nbytes, ctypes.byref(h))
    return st, h


@pytest.mark.parametrize("kw,status", [
    (dict(S=0), 2), (dict(S=2000), 2), (dict(d_in=12), 2), (dict(d_out=0), 2),
    (dict(d_in=1 << 20), 2), (dict(w=7), 3), (dict(meta=0), 1), (dict(meta=FAKE_ODD), 4),
    (dict(nbytes=16), 8),
])
def test_table_create_rejects(kw, status):
    st, h = _create(**kw)
    assert st == status
    assert h.value is None
    assert lora.lib().lora_last_error()


def test_table_set_and_clear_validation():
    L = lora.lib()
    st, h = _create()
    assert st == 0
    A = ctypes.c_void_p(FAKE)
    assert L.lora_table_set(h, 0, 16, 2.0, A, A) == 0
    assert L.lora_table_set(h, 4, 16, 2.0, A, A) == 6          # slot out of range
    assert L.lora_table_set(h, -1, 16, 2.0, A, A) == 6
    assert L.lora_table_set(h, 1, 0, 2.0, A, A) == 5           # rank 0
    assert L.lora_table_set(h, 1, 129, 2.0, A, A) == 5         # rank > max
    assert L.lora_table_set(h, 1, 8, 2.0, None, A) == 1
    assert L.lora_table_set(h, 1, 8, 2.0, ctypes.c_void_p(FAKE_ODD), A) == 4
    assert L.lora_table_clear(h, 0) == 0
    assert L.lora_table_clear(h, 9) == 6
    assert L.lora_table_set(None, 0, 8, 1.0, A, A) == 1
    L.lora_table_destroy(h)


def test_plan_build_validation():
    L = lora.lib()
    st, t = _create(S=8)
    assert st == 0
    need = L.lora_plan_workspace_bytes(100, 8)
    assert need > 0 and L.lora_plan_workspace_bytes(200, 8) > need
    p = ctypes.c_void_p()
    ws = ctypes.c_void_p(FAKE)
    idx = ctypes.c_void_p(FAKE)
    assert L.lora_plan_build(t, -1, idx, None, ws, need, None, ctypes.byref(p)) == 2
    assert L.lora_plan_build(t, (1 << 22) + 1, idx, None, ws, 1 << 40, None, ctypes.byref(p)) == 2
    assert L.lora_plan_build(t, 100, idx, None, ws, need - 1, None, ctypes.byref(p)) == 8
    assert L.lora_plan_build(t, 100, None, None, ws, need, None, ctypes.byref(p)) == 1
    assert L.lora_plan_build(t, 100, idx, None, None, need, None, ctypes.byref(p)) == 1
    assert L.lora_plan_build(t, 100, ctypes.c_void_p(FAKE + 2), None, ws, need, None,
                             ctypes.byref(p)) == 4
    assert L.lora_plan_build(None, 100, idx, None, ws, need, None, ctypes.byref(p)) == 1
    assert L.lora_plan_build_segments(t, 100, 3, None, idx, None, ws, need, None,
                                      ctypes.byref(p)) == 1
    assert L.lora_plan_build_segments(t, 100, -1, idx, idx, None, ws, need, None,
                                      ctypes.byref(p)) == 2
    assert p.value is None
    L.lora_table_destroy(t)


@pytest.mark.parametrize("field,value", [
    ("small_max", -2), ("small_split", 2), ("split_slices", 0), ("split_slices", 9),
    ("small_chunks", 17), ("fork", 3), ("grad_splits", 0), ("grad_splits", 9),
    ("block_rows", 0), ("block_rows", 128),
])
def test_plan_policy_validation(field, value):
    """A path policy outside its documented range is refused on the host
    (LORA_ERR_VALUE) before anything is enqueued; the defaults are all -1."""
    L = lora.lib()
    st, t = _create(S=8)
    assert st == 0
    q = lora.Policy()
    assert [getattr(q, f) for f, _ in lora.Policy._fields_] == [-1] * len(lora.Policy._fields_)
    setattr(q, field, value)
    p = ctypes.c_void_p()
    need = L.lora_plan_workspace_bytes(100, 8)
    assert L.lora_plan_build_policy(t, 100, ctypes.c_void_p(FAKE), None, ctypes.byref(q),
                                    ctypes.c_void_p(FAKE), need, None, ctypes.byref(p)) == 10
    assert p.value is None
    assert field.encode() in L.lora_last_error()
    L.lora_table_destroy(t)


def test_plan_workspace_does_not_depend_on_policy():
    """The plan workspace size is a function of n and num_slots alone."""
    L = lora.lib()
    sizes = {n: L.lora_plan_workspace_bytes(n, 33) for n in (0, 1, 100, 1024, 1025, 5000, 70000)}
    assert all(v > 0 for v in sizes.values())
    assert sizes[1025] > sizes[1024] and sizes[70000] > sizes[5000]


def test_library_reads_no_environment():
    """No process-wide switches: neither the sources nor the built library
    call getenv (path selection is per plan, through lora_policy)."""
    csrc = os.path.join(ROOT, "paper_2601_07376_amd", "csrc")
    for f in os.listdir(csrc):
        text = open(os.path.join(csrc, f)).read()
        assert "getenv" not in text, f"{f} reads the environment"
    for path in (lora.LIB_PATH, lora.DEBUG_LIB_PATH):
        if os.path.exists(path):
            assert b"getenv" not in open(path, "rb").read(), path


def test_ops_reject_null_plan():
    L = lora.lib()
    X = ctypes.c_void_p(FAKE)
    assert L.lora_shrink(None, X, 1, 64, X, 16, None) == 1
    assert L.lora_expand(None, X, 16, X, 1, 64, None) == 1
    assert L.lora_apply(None, X, 1, 64, X, 1, 64, X, 1 << 20, None) == 1
    assert L.lora_grad(None, X, 1, 64, X, 1, 64, None, 0, None, None, 0, X, 1 << 20, None) == 1
    assert L.lora_plan_check(None, None, None) == 1
    assert L.lora_plan_export(None, *([None] * 11), None) == 1
    assert L.lora_apply_workspace_bytes(None) == 0
    assert L.lora_grad_workspace_bytes(None) == 0


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(lora, "_libs", {})
    monkeypatch.setattr(lora, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(lora, "DEBUG_LIB_PATH", str(tmp_path / "missing_debug.so"))
    with pytest.raises(RuntimeError, match="missing"):
        lora.lib()
    with pytest.raises(RuntimeError, match="missing"):
        lora.lib(debug=True)


def _adam(**kw):
    base = dict(p=FAKE, m=FAKE + 0x1000, v=FAKE + 0x2000, g=FAKE + 0x3000, p_bf16=FAKE + 0x4000,
                n=256, step=1, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01)
    base.update(kw)
    return lora.AdamWTensor(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(step=0), 10), (dict(lr=-1.0), 10), (dict(lr=float("nan")), 10), (dict(beta1=1.0), 10),
    (dict(beta2=-0.1), 10), (dict(eps=0.0), 10), (dict(weight_decay=float("inf")), 10),
    (dict(n=-1), 2), (dict(p=0), 1), (dict(g=0), 1), (dict(m=FAKE_ODD), 4),
    (dict(p_bf16=FAKE + 0x4008), 4),
    (dict(m=FAKE + 0x200), 2),                 # m overlaps p (n = 256 floats = 1 KiB)
    (dict(p_bf16=FAKE + 0x3100), 2),           # the bf16 copy overlaps the gradient
])
def test_adamw_rejects(kw, status):
    """Host validation only: every record is rejected before anything is enqueued."""
    L = lora.lib()
    recs = (lora.AdamWTensor * 1)(_adam(**kw))
    assert L.lora_adamw_step(ctypes.cast(recs, ctypes.c_void_p), 1, None) == status
    assert L.lora_last_error()


def test_adamw_count_and_cross_record_overlap():
    L = lora.lib()
    recs = (lora.AdamWTensor * 2)(_adam(), _adam(p=FAKE + 0x10000, m=FAKE + 0x11000,
                                                 v=FAKE + 0x12000, g=FAKE + 0x13000,
                                                 p_bf16=FAKE + 0x2100))   # into record 0's v
    assert L.lora_adamw_step(ctypes.cast(recs, ctypes.c_void_p), 2, None) == 2
    assert L.lora_adamw_step(ctypes.cast(recs, ctypes.c_void_p), -1, None) == 2
    assert L.lora_adamw_step(None, 1, None) == 1
    assert L.lora_adamw_step(None, 0, None) == 0        # nothing to do
    # a zero-size record is skipped (nothing to validate but its hyperparameters)
    empty = (lora.AdamWTensor * 1)(_adam(n=0, p=0, m=0, v=0, g=0, p_bf16=0))
    assert L.lora_adamw_step(ctypes.cast(empty, ctypes.c_void_p), 1, None) == 0


def _loss_call(kind=0, n=4, vocab=64, z=FAKE, ldz=64, target=FAKE + 0x8000, weight=FAKE + 0x9000,
               old=FAKE + 0xa000, adv=FAKE + 0xb000, clip_lo=0.2, loss=FAKE + 0xc000,
               dz=FAKE + 0x20000, ldd=64):
    L = lora.lib()
    v = lambda x: ctypes.c_void_p(x) if x else None
    return L.lora_token_loss(kind, n, vocab, v(z), lora.LORA_BF16, ldz, v(target), v(weight), None,
                             v(old), v(adv), None, clip_lo, 0.2, v(loss), None, v(dz),
                             lora.LORA_F32, ldd, None)


@pytest.mark.parametrize("kw,status", [
    (dict(kind=7), 10), (dict(n=-1), 2), (dict(vocab=0), 2), (dict(clip_lo=-0.5), 10),
    (dict(clip_lo=float("nan")), 10), (dict(z=FAKE_ODD), 4), (dict(ldz=60), 2), (dict(ldd=68), 4),
    (dict(z=0), 1), (dict(target=0), 1), (dict(loss=0), 1), (dict(weight=0), 1),
    (dict(kind=2, adv=0), 1), (dict(dz=FAKE + 0x100), 2),      # dlogits overlaps logits
])
def test_token_loss_rejects(kw, status):
    """Host validation only: every call here is rejected before anything is enqueued."""
    assert _loss_call(**kw) == status
    assert lora.lib().lora_last_error()


def test_token_loss_empty_batch():
    assert _loss_call(n=0, target=0, loss=0, weight=0) == 0


def test_backward_rejects_null_plan():
    L = lora.lib()
    assert L.lora_backward_workspace_bytes(None) == 0
    st = L.lora_backward(None, ctypes.c_void_p(FAKE), lora.LORA_BF16, 64, ctypes.c_void_p(FAKE),
                         lora.LORA_BF16, 64, None, 0, None, None, 0, ctypes.c_void_p(FAKE),
                         lora.LORA_F32, 64, ctypes.c_void_p(FAKE), 1 << 20, None)
    assert st == 1 and L.lora_last_error()


def test_apply_ids_validation():
    """lora_apply_ids refuses bad arguments on the host, before anything is
    enqueued; its workspace is 0 bytes for n = 0 or a table without adapters,
    and grows with n and the slices x rank tiles of the live ranks."""
    L = lora.lib()
    st, h = _create(S=4, d_in=1024, d_out=512)
    assert st == 0
    F = ctypes.c_void_p(FAKE)
    assert L.lora_apply_ids_workspace_bytes(h, 100) == 0          # no adapter yet
    assert L.lora_table_set(h, 0, 16, 2.0, F, F) == 0
    need = L.lora_apply_ids_workspace_bytes(h, 100)
    assert need == 4 * 100 * 16 * 4                                # 4 d-slices x n x 16 floats
    assert L.lora_table_set(h, 2, 40, 1.0, F, F) == 0
    assert L.lora_apply_ids_workspace_bytes(h, 100) == 4 * 100 * 64 * 4
    assert L.lora_apply_ids_workspace_bytes(h, 0) == 0
    assert L.lora_apply_ids_workspace_bytes(h, 1025) == 0
    assert L.lora_apply_ids_workspace_bytes(None, 100) == 0
    need = L.lora_apply_ids_workspace_bytes(h, 100)
    args = lambda **kw: dict(dict(t=h, n=100, idx=F, X=F, xd=lora.LORA_BF16, ldx=1024, Y=F,
                                  yd=lora.LORA_F32, ldy=512, ws=F, nb=need), **kw)
    call = lambda a: L.lora_apply_ids(a["t"], a["n"], a["idx"], a["X"], a["xd"], a["ldx"], a["Y"],
                                      a["yd"], a["ldy"], a["ws"], a["nb"], None)
    assert call(args(t=None)) == 1
    assert call(args(n=1025)) == 2
    assert call(args(n=-1)) == 2
    assert call(args(xd=lora.LORA_F32)) == 3
    assert call(args(idx=None)) == 1
    assert call(args(idx=ctypes.c_void_p(FAKE_ODD))) == 4
    assert call(args(X=None)) == 1
    assert call(args(ldx=1000)) in (2, 4)
    assert call(args(ws=None)) == 1
    assert call(args(ws=ctypes.c_void_p(FAKE_ODD))) == 4
    assert call(args(nb=need - 1)) == 8
    assert b"workspace" in L.lora_last_error()
    L.lora_table_destroy(h)
