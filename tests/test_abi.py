"""Host-only checks of the C-ABI library: it loads, exports every entry point that
include/clsa.h declares, and rejects bad arguments before touching the GPU."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "clsa.h")
LIB = os.path.join(ROOT, "paper_2606_06467_amd", "libclsa.so")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_2606_06467_amd import _build
        _build.build()
    from paper_2606_06467_amd import binding
    return binding.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(clsa_[a-z_]+)\s*\(", text)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("clsa_index_scores", "clsa_topk", "clsa_sparse_attn", "clsa_decode_step",
              "clsa_decode_step_grouped", "clsa_dense_attn", "clsa_project_append",
              "clsa_kd_target", "clsa_kd_loss", "clsa_workspace_bytes",
              "clsa_status_string", "clsa_set_phase_events", "clsa_get_device_error"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT (clsa_\w+)", out))
    missing = [n for n in declared_functions() if n not in exported]
    assert not missing, missing
    for n in declared_functions():
        assert hasattr(lib, n)


def test_library_is_gfx950_only(lib, tmp_path):
    """The device code bundled into the library targets gfx950 and nothing else."""
    fb = tmp_path / "fatbin"
    subprocess.run(["objcopy", f"--dump-section=.hip_fatbin={fb}", LIB, str(tmp_path / "x.so")],
                   check=True)
    out = subprocess.run(["/opt/rocm/llvm/bin/clang-offload-bundler", "--list", "--type=o",
                          f"--input={fb}"], capture_output=True, text=True, check=True)
    targets = [t for t in out.stdout.split() if "amdgcn" in t]
    assert targets and all(t.endswith("gfx950") for t in targets), targets


def test_status_strings(lib):
    from paper_2606_06467_amd import binding as B
    assert B.clsa_status_string(0) == "CLSA_OK"
    assert B.clsa_status_string(-1) == "CLSA_ERR_INVALID_ARG"
    assert B.clsa_status_string(-2) == "CLSA_ERR_UNSUPPORTED"
    assert B.clsa_status_string(-3) == "CLSA_ERR_WORKSPACE"
    assert B.clsa_status_string(-4) == "CLSA_ERR_HIP"
    assert B.clsa_status_string(7) == "CLSA_ERR_UNKNOWN"


# Fake, aligned, never-dereferenced device addresses: every call below must be
# rejected by host validation before anything is enqueued.
A = ctypes.c_void_p(0x10000)
MIS = ctypes.c_void_p(0x10002)


def _shape(**kw):
    from paper_2606_06467_amd import binding as B
    base = dict(batch=2, n_q=1, max_len=1024, top_k=64)
    base.update(kw)
    return B.make_shape(**base)


def _index(lib, sh, q=A, k=A, pt=None, sl=A, qp=None, sc=A):
    return lib.clsa_index_scores(ctypes.byref(sh), q, k, pt, sl, qp, sc, None)


def _attn(lib, sh, q=A, k=A, v=A, pt=None, idx=A, ns=A, out=A, lse=None, ws=None, wsb=0):
    return lib.clsa_sparse_attn(ctypes.byref(sh), q, k, v, pt, idx, ns, out, lse, ws, wsb, None)


def _step(lib, sh, ws=None, wsb=0, L=2, **kw):
    a = dict(q_idx=A, k_idx=A, k=A, v=A, pt=None, sl=A, qp=None, ql=A, ol=A, lse=None, idx=A, ns=A)
    a.update(kw)
    return lib.clsa_decode_step(ctypes.byref(sh), a["q_idx"], a["k_idx"], a["k"], a["v"], a["pt"],
                                a["sl"], a["qp"], L, a["ql"], a["ol"], a["lse"], a["idx"], a["ns"],
                                ws, wsb, None)


@pytest.mark.parametrize("field,value,code", [
    ("batch", 0, -1), ("n_q", 0, -1), ("max_len", 0, -1), ("top_k", 0, -1), ("top_k", -5, -1),
    ("idx_heads", 0, -1), ("causal", 2, -1), ("page_size", 48, -1), ("page_size", -64, -1),
    ("idx_dim", 32, -2), ("top_k", 8193, -2), ("max_len", 262144 * 2, -2),
])
def test_index_rejects_bad_shapes(lib, field, value, code):
    sh = _shape(**{field: value})
    assert _index(lib, sh) == code


def test_index_rejects_bad_pointers(lib):
    sh = _shape()
    assert _index(lib, sh, q=None) == -1
    assert _index(lib, sh, q=MIS) == -1       # bf16 tensors need 16-byte alignment
    assert _index(lib, sh, k=None) == -1
    assert _index(lib, sh, sl=None) == -1
    assert _index(lib, sh, sc=None) == -1
    assert _index(lib, _shape(causal=True), qp=None) == -1              # causal needs q_pos
    assert _index(lib, _shape(page_size=64, max_pages=16), pt=None) == -1
    assert _index(lib, _shape(page_size=64, max_pages=15), pt=A) == -1  # table too narrow
    assert _index(lib, _shape(page_size=64, max_pages=16, max_len=1000), pt=A) == -1
    assert _index(lib, _shape(page_size=8, max_pages=128), pt=A) == -2


@pytest.mark.parametrize("kw,code", [
    (dict(head_dim=64), -2), (dict(q_heads=32, kv_heads=5), -1), (dict(q_heads=48, kv_heads=8), -2),
    (dict(q_heads=20, kv_heads=4), None), (dict(softmax_scale=float("nan")), -1),
    (dict(softmax_scale=float("inf")), -1),
    # one contiguous sequence's cache of 4 GiB: beyond the 32-bit offsets
    (dict(max_len=262144, q_heads=64, kv_heads=64), -2),
    (dict(max_len=262143, q_heads=64, kv_heads=64), None),
])
def test_attn_rejects_bad_shapes(lib, kw, code):
    from paper_2606_06467_amd import binding as B
    sh = _shape(top_k=2048, **kw)
    if code is None:
        # supported shape: it needs a workspace (so the call below cannot reach a
        # launch with the fake pointers) and fails only on the missing workspace
        assert B.clsa_workspace_bytes(sh, B.CLSA_OP_ATTN) > 0
        assert _attn(lib, sh, ws=None, wsb=0) == -3
    else:
        assert _attn(lib, sh, ws=None, wsb=0) == code


def test_attn_pointer_and_workspace_checks(lib):
    from paper_2606_06467_amd import binding as B
    sh = _shape(top_k=2048)
    need = B.clsa_workspace_bytes(sh, B.CLSA_OP_ATTN)
    assert need > 0 and need % 256 == 0
    assert _attn(lib, sh, q=MIS) == -1
    assert _attn(lib, sh, out=None) == -1
    assert _attn(lib, sh, lse=ctypes.c_void_p(0x10001)) == -1
    assert _attn(lib, sh, ws=None, wsb=need) == -3
    assert _attn(lib, sh, ws=A, wsb=need - 1) == -3
    assert _attn(lib, sh, ws=ctypes.c_void_p(0x10010), wsb=need) == -3   # not 256-byte aligned


def test_decode_step_checks(lib):
    from paper_2606_06467_amd import binding as B
    sh = _shape()
    need = B.clsa_workspace_bytes(sh, B.CLSA_OP_DECODE, 2)
    assert need >= 2 * 1024 * 4
    assert _step(lib, sh, ws=None, wsb=need) == -3
    assert _step(lib, sh, ws=A, wsb=need - 256) == -3
    assert _step(lib, sh, ws=A, wsb=need, L=-1) == -1
    assert _step(lib, sh, ws=A, wsb=need, q_idx=None) == -1
    assert _step(lib, sh, ws=A, wsb=need, ql=None) == -1
    assert _step(lib, sh, ws=A, wsb=need, idx=None) == -1
    assert _step(lib, _shape(causal=True), ws=A, wsb=need) == -1
    assert _step(lib, _shape(head_dim=96), ws=A, wsb=need) == -2


def test_workspace_sizes(lib):
    from paper_2606_06467_amd import binding as B
    sh = _shape(batch=4, max_len=131072, top_k=2048)
    assert B.clsa_workspace_bytes(sh, B.CLSA_OP_INDEX) == 0
    # few rows: the multi-workgroup top-k keeps bitmaps and candidates in the workspace
    assert B.clsa_workspace_bytes(sh, B.CLSA_OP_TOPK) >= 2 * 4 * 131072 // 8
    # many rows: one workgroup per row, everything in LDS
    many = _shape(batch=1, n_q=4096, max_len=131072, top_k=2048, causal=True)
    assert B.clsa_workspace_bytes(many, B.CLSA_OP_TOPK) == 0
    # many rows: every index list in 8 stretches, fp32 (o, m, l) partials per stretch
    assert B.clsa_workspace_bytes(many, B.CLSA_OP_ATTN) >= 4096 * 32 * 8 * 130 * 4
    few = _shape(batch=1, n_q=64, max_len=131072, top_k=2048, causal=True)
    assert B.clsa_workspace_bytes(few, B.CLSA_OP_ATTN) > 0           # split over the list
    dec = B.clsa_workspace_bytes(sh, B.CLSA_OP_DECODE, 16)
    assert dec >= 4 * 131072 * 4 + 4 * 2048 * 4
    assert dec == B.clsa_workspace_bytes(sh, B.CLSA_OP_DECODE, 1)   # layers reuse buffers
    assert B.clsa_workspace_bytes(sh, B.CLSA_OP_DECODE, -1) == 0
    assert B.clsa_workspace_bytes(_shape(top_k=0), B.CLSA_OP_DECODE, 1) == 0
    assert B.clsa_workspace_bytes(sh, 99) == 0


def test_phase_event_hook_arguments(lib):
    from paper_2606_06467_amd import binding as B
    assert lib.clsa_set_phase_events(None, 0) == 0
    assert lib.clsa_set_phase_events(None, 4) == -1
    arr = (ctypes.c_void_p * 3)(A, A, A)
    assert lib.clsa_set_phase_events(arr, 3) == -1
    arr4 = (ctypes.c_void_p * 4)(A, A, None, A)
    assert lib.clsa_set_phase_events(arr4, 4) == -1
    many = (ctypes.c_void_p * (4 + 2 * 65))(*([A] * (4 + 2 * 65)))
    assert lib.clsa_set_phase_events(many, 5) == -1              # odd: pairs per layer
    assert lib.clsa_set_phase_events(many, 4 + 2 * 65) == -1     # at most 64 layers
    assert lib.clsa_set_phase_events(many, 4 + 2 * 64) == 0
    assert lib.clsa_set_phase_events(many, 6) == 0
    assert lib.clsa_set_phase_events(None, 0) == 0


def test_get_device_error_rejects_null(lib):
    assert lib.clsa_get_device_error(None) == -1


def _symbols():
    out = subprocess.run(["readelf", "-sW", LIB], capture_output=True, text=True, check=True).stdout
    return [line.split() for line in out.splitlines() if len(line.split()) >= 8]


def test_phase_hook_is_thread_local():
    """The profiling hook is per host thread: its storage is a TLS object, so
    calls from other threads never read or write it."""
    hooks = [f for f in _symbols() if "hook" in f[7]]
    assert hooks and all(f[3] == "TLS" for f in hooks), hooks


def test_no_function_static_state_in_the_entry_points():
    """Host-side mutable state of the entry points: no function-local statics
    (``_ZZ`` symbols), and of the file-scope objects of the host code only the
    per-device property cache (an array of atomics indexed by device) is a
    non-TLS object."""
    syms = _symbols()
    assert not [f[7] for f in syms if f[7].startswith("_ZZ")]
    objs = [f[7] for f in syms if f[3] == "OBJECT" and "GLOBAL__N" in f[7]]
    assert objs and all("lds_limit" in n for n in objs), objs


def test_phase_hook_set_from_threads(lib):
    """Setting and clearing the hook from many threads at once is safe (each
    thread writes only its own copy) and every call reports the same status."""
    import threading
    arr = (ctypes.c_void_p * 6)(A, A, A, A, A, A)
    res = []

    def work():
        r = []
        for i in range(200):
            r.append(lib.clsa_set_phase_events(arr, 6 if i % 2 == 0 else 4))
            r.append(lib.clsa_set_phase_events(None, 0))
        res.append(r)

    th = [threading.Thread(target=work) for _ in range(8)]
    for t in th:
        t.start()
    for t in th:
        t.join()
    assert len(res) == 8 and all(v == 0 for r in res for v in r)


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    from paper_2606_06467_amd import binding as B
    monkeypatch.setattr(B, "_lib_handle", None)
    monkeypatch.setattr(B, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="no fallback"):
        B.lib()


def _grouped_call(lib, sh, ws=A, wsb=1 << 30, group=1, sq=0, sk=0, L=2):
    return lib.clsa_decode_step_grouped(ctypes.byref(sh), A, sq, A, sk, A, A, None, A, None, L,
                                        group, A, A, None, A, A, ws, wsb, None)


def test_grouped_step_checks(lib):
    sh = _shape()
    assert _grouped_call(lib, sh, group=0) == -1
    assert _grouped_call(lib, sh, group=-3) == -1
    assert _grouped_call(lib, sh, sq=4) == -1          # set strides keep 16-byte alignment
    assert _grouped_call(lib, sh, sk=-8) == -1
    assert _grouped_call(lib, sh, L=-1) == -1
    assert _grouped_call(lib, sh, ws=None) == -3
    assert _grouped_call(lib, _shape(head_dim=64)) == -2


def test_dense_attn_checks(lib):
    from paper_2606_06467_amd import binding as B
    def call(sh, ws=None, wsb=0, q=A, sl=A, qp=None):
        return lib.clsa_dense_attn(ctypes.byref(sh), q, A, A, None, sl, qp, A, None, ws, wsb, None)
    sh = _shape(batch=4, max_len=131072, top_k=2048)
    need = B.clsa_workspace_bytes(sh, B.CLSA_OP_DENSE)
    assert need > B.clsa_workspace_bytes(sh, B.CLSA_OP_ATTN)   # splits over every key
    assert call(sh, ws=None, wsb=0) == -3
    assert call(sh, ws=A, wsb=need - 1) == -3
    assert call(sh, ws=A, wsb=need, q=MIS) == -1
    assert call(sh, ws=A, wsb=need, sl=None) == -1
    assert call(_shape(causal=True), ws=A, wsb=1 << 30) == -1      # causal needs q_pos
    assert call(_shape(max_len=262144 * 2), ws=A, wsb=1 << 30) == -2
    assert call(_shape(head_dim=96), ws=A, wsb=1 << 30) == -2
    assert B.clsa_workspace_bytes(_shape(max_len=262144 * 2), B.CLSA_OP_DENSE) == 0


def test_project_append_checks(lib):
    def call(sh, d=2560, h=A, w=A, pos=A, pt=None):
        return lib.clsa_project_append(ctypes.byref(sh), d, h, w, pos, pt, A, A, A, A, None)
    sh = _shape()
    assert call(sh, d=0) == -1
    assert call(sh, d=2500) == -2          # not a multiple of 512
    assert call(sh, d=8704) == -2          # above 8192
    assert call(sh, h=MIS) == -1
    assert call(sh, w=None) == -1
    assert call(sh, pos=None) == -1
    assert call(_shape(page_size=64, max_pages=16), pt=None) == -1
    assert call(_shape(idx_dim=32)) == -2
    assert call(_shape(head_dim=64)) == -2


def test_kd_target_checks(lib):
    from paper_2606_06467_amd import binding as B
    def call(sh, L=4, ws=A, wsb=1 << 30, ql=A, kc=A, sl=A, qp=None, ab=A, lse=None):
        return lib.clsa_kd_target(ctypes.byref(sh), L, ql, kc, None, sl, qp, lse, ab, ws, wsb,
                                  None)
    sh = _shape(n_q=128, max_len=4096)
    need = B.clsa_workspace_bytes(sh, B.CLSA_OP_KD_TARGET, 4)
    assert need >= 4 * 128 * 32 * 4                       # one lse per (layer, row, head)
    assert need > B.clsa_workspace_bytes(sh, B.CLSA_OP_KD_TARGET, 2)
    assert B.clsa_workspace_bytes(sh, B.CLSA_OP_KD_TARGET, 0) == 0
    assert call(sh, L=0) == -1
    assert call(sh, ws=None, wsb=0) == -3
    assert call(sh, wsb=need - 1) == -3
    assert call(sh, ws=MIS, wsb=need) == -3                # workspace must be 256-byte aligned
    assert call(sh, ql=MIS) == -1
    assert call(sh, kc=None) == -1
    assert call(sh, sl=None) == -1
    assert call(sh, ab=None) == -1
    assert call(sh, lse=MIS) == -1                         # optional lse: 4-byte aligned
    assert call(_shape(n_q=128, max_len=4096, causal=True)) == -1        # causal needs q_pos
    assert call(_shape(page_size=64, max_pages=16)) == -1                 # paged needs a table
    assert call(_shape(head_dim=64)) == -2
    assert call(_shape(q_heads=32, kv_heads=3)) == -1
    neg = _shape()
    neg.softmax_scale = -0.1
    assert call(neg) == -1


def test_kd_loss_checks(lib):
    from paper_2606_06467_amd import binding as B
    def call(sh, ws=A, wsb=1 << 40, ab=A, qi=A, ki=A, sl=A, qp=None, loss=A, dq=A, dk=A):
        return lib.clsa_kd_loss(ctypes.byref(sh), ab, qi, ki, None, sl, qp, loss, dq, dk, ws, wsb,
                                None)
    sh = _shape(n_q=128, max_len=4096)
    need = B.clsa_workspace_bytes(sh, B.CLSA_OP_KD_LOSS)
    assert need >= 128 * 4096 * 4                          # scores, then dL/dI, per row and key
    assert call(sh, ws=None, wsb=0) == -3
    assert call(sh, wsb=need - 1) == -3
    assert call(sh, ab=None) == -1
    assert call(sh, qi=MIS) == -1
    assert call(sh, ki=None) == -1
    assert call(sh, loss=None) == -1
    assert call(sh, dq=MIS) == -1                          # fp32 gradients in 16-byte vectors
    assert call(sh, dk=None) == -1
    assert call(_shape(n_q=128, max_len=4096, causal=True)) == -1
    assert call(_shape(idx_dim=32)) == -2
    assert call(_shape(max_len=262144 * 2)) == -2
    assert B.clsa_workspace_bytes(_shape(idx_dim=32), B.CLSA_OP_KD_LOSS) == 0
