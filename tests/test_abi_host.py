"""Host-side checks of the C ABI (no GPU): the library loads, exports every
function declared in include/attn_mi355x.h, and every validation error is
returned before anything reaches the GPU."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "attn_mi355x.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(attn_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    import paper_2609_33916_amd as pkg
    if not os.path.exists(pkg.LIB_PATH):
        pytest.fail("libattn_mi355x.so is not built (python -m paper_2609_33916_amd.build)")
    return pkg.lib()


def test_exports_every_declared_function(L):
    names = _declared_functions()
    assert set(names) >= {"attn_fwd", "attn_fwd_bwd", "attn_workspace_bytes", "attn_strerror"}
    for name in names:
        assert hasattr(L, name), name


def test_workspace_bytes(L):
    assert L.attn_workspace_bytes(2, 32, 16384, 128) == 2 * 2 * 32 * 16384 * 4
    assert L.attn_workspace_bytes(1, 1, 1, 32) == 8
    assert L.attn_workspace_bytes(0, 1, 1, 32) == 0
    assert L.attn_workspace_bytes(1, 1, -5, 32) == 0


def test_strerror(L):
    import paper_2609_33916_amd as pkg
    for code in range(0, -9, -1):
        s = pkg.attn_strerror(code)
        assert s and "unknown" not in s
    assert "unknown" in pkg.attn_strerror(12345)


FAKE = 1 << 20          # aligned, never dereferenced: validation fails first
MIS = FAKE + 2          # misaligned


def _fwd(L, Q=FAKE, K=FAKE, V=FAKE, O=FAKE, Lse=FAKE, B=1, H=1, n=8, d=64, scale=0.125,
         causal=0, dtype=0):
    return L.attn_fwd(Q, K, V, O, Lse, B, H, n, d, scale, causal, dtype, None)


def _fb(lib_, ws=FAKE, wsb=1 << 30, B=1, H=1, n=8, d=64, scale=0.125, causal=0, dtype=1, **ptr):
    p = {k: FAKE for k in ("Q", "K", "V", "dO", "O", "L", "dQ", "dK", "dV")}
    p.update(ptr)
    return lib_.attn_fwd_bwd(p["Q"], p["K"], p["V"], p["dO"], p["O"], p["L"], p["dQ"], p["dK"],
                          p["dV"], ws, wsb, B, H, n, d, scale, causal, dtype, None)


def test_fwd_validation(L):
    assert _fwd(L, Q=None) == -1
    assert _fwd(L, Lse=None) == -1
    assert _fwd(L, B=0) == -2
    assert _fwd(L, n=0) == -2
    assert _fwd(L, H=-1) == -2
    assert _fwd(L, d=80) == -3
    assert _fwd(L, d=256) == -3
    assert _fwd(L, dtype=7) == -3
    assert _fwd(L, scale=float("nan")) == -7
    assert _fwd(L, scale=float("inf")) == -7
    assert _fwd(L, causal=2) == -7
    assert _fwd(L, V=MIS) == -4
    assert _fwd(L, Lse=FAKE + 2) == -4
    assert _fwd(L, n=1 << 25, d=128) == -2   # n*d beyond 32-bit indexing


def test_fwd_bwd_validation(L):
    for name in ("Q", "K", "V", "dO", "O", "L", "dQ", "dK", "dV"):
        assert _fb(L, **{name: None}) == -1, name
    assert _fb(L, ws=None) == -1
    for name in ("Q", "K", "V", "dO", "O", "dQ", "dK", "dV"):
        assert _fb(L, **{name: MIS}) == -4, name
    assert _fb(L, ws=FAKE + 1) == -4
    assert _fb(L, wsb=2 * 8 * 4 - 1) == -5
    assert _fb(L, d=48) == -3
    assert _fb(L, dtype=-1) == -3
    assert _fb(L, B=0) == -2
    assert _fb(L, scale=float("-inf")) == -7
    assert _fb(L, causal=-1) == -7


def test_bwd_validation(L):
    def call(**kw):
        p = {k: FAKE for k in ("Q", "K", "V", "O", "L", "dO", "dQ", "dK", "dV", "ws")}
        p.update(kw)
        return L.attn_bwd(p["Q"], p["K"], p["V"], p["O"], p["L"], p["dO"], p["dQ"], p["dK"],
                          p["dV"], p["ws"], kw.get("wsb", 1 << 30), 1, 1, 8, 64, 0.125, 0, 0, None)
    for name in ("Q", "K", "V", "O", "L", "dO", "dQ", "dK", "dV", "ws"):
        assert call(**{name: None}) == -1, name
    for name in ("Q", "K", "V", "O", "dO", "dQ", "dK", "dV"):
        assert call(**{name: MIS}) == -4, name
    assert call(wsb=1) == -5


def test_atomic_validation(L):
    assert L.attn_workspace_bytes_atomic(2, 3, 100, 64) == 2 * 3 * 100 * (64 * 4 + 8)
    assert L.attn_workspace_bytes_atomic(1, 1, 1, 48) == 0

    def call(dtype=0, ws=FAKE, wsb=1 << 30, **kw):
        p = {k: FAKE for k in ("Q", "K", "V", "dO", "O", "L", "dQ", "dK", "dV")}
        p.update(kw)
        return L.attn_fwd_bwd_atomic(p["Q"], p["K"], p["V"], p["dO"], p["O"], p["L"], p["dQ"], p["dK"],
                                     p["dV"], ws, wsb, 1, 2, 9, 64, 0.125, 1, dtype, None)
    assert call(dtype=1) == -3            # bfloat16 only
    assert call(ws=None) == -1
    assert call(ws=FAKE + 4) == -4        # the accumulator needs 16-byte alignment
    assert call(wsb=2 * 9 * (64 * 4 + 8) - 1) == -5
    for name in ("Q", "K", "V", "dO", "O", "L", "dQ", "dK", "dV"):
        assert call(**{name: None}) == -1, name


def test_decode_validation(L):
    # no split at 300 keys for 16 groups? workspace only when the keys are split
    assert L.attn_decode_workspace_bytes(1, 8, 1, 50000, 128, 1) > 0
    assert L.attn_decode_workspace_bytes(64, 64, 8, 100, 128, 1) == 0
    assert L.attn_decode_workspace_bytes(1, 6, 4, 10, 64, 1) == 0      # 6 % 4 != 0: invalid

    def call(q=FAKE, kn=FAKE, vn=FAKE, kc=FAKE, vc=FAKE, lens=None, o=FAKE, lse=FAKE, ws=FAKE, wsb=1 << 30,
             B=2, Hq=8, Hkv=2, n=10, n_cap=11, d=64, scale=0.125, dtype=0):
        return L.attn_decode(q, kn, vn, kc, vc, lens, o, lse, ws, wsb, B, Hq, Hkv, n, n_cap, d, scale, dtype, None)
    assert call(q=None) == -1
    assert call(kc=None) == -1
    assert call(o=None) == -1
    assert call(kn=None) == -1             # k_new without v_new
    assert call(n_cap=10) == -2           # no room for the appended row
    assert call(kn=None, vn=None, n_cap=9) == -2    # without an append n_cap must still hold n rows
    assert call(Hq=6, Hkv=4) == -2
    assert call(Hkv=0) == -2
    assert call(n=-1) == -2
    assert call(d=80) == -3
    assert call(dtype=1) == -3            # bfloat16 only
    assert call(scale=float("nan")) == -7
    assert call(q=MIS) == -4
    assert call(lens=FAKE + 2) == -4
    assert call(lse=FAKE + 2) == -4
    big = dict(B=1, Hq=8, Hkv=1, n=50000, n_cap=50001, d=128)
    assert call(ws=None, **big) == -1
    assert call(ws=FAKE + 4, **big) == -4
    assert call(wsb=16, **big) == -5


def test_mat_bytes(L):
    # [B, H, n, lda] with lda = n rounded up to 128
    assert L.attn_mat_bytes(2, 3, 100, 0) == 2 * 3 * 100 * 128 * 2
    assert L.attn_mat_bytes(1, 1, 128, 1) == 128 * 128 * 4
    assert L.attn_mat_bytes(1, 1, 129, 1) == 129 * 256 * 4
    assert L.attn_mat_bytes(128, 1, 4096, 0) == 128 * 4096 * 4096 * 2
    assert L.attn_mat_bytes(1, 1, 0, 0) == 0
    assert L.attn_mat_bytes(1, 1, 8, 5) == 0
    assert L.attn_mat_bytes(1, 1, (1 << 20) + 1, 0) == 0


def test_mat_validation(L):
    P_OK = 1 << 40

    def fwd(P=FAKE, pb=P_OK, n=8, **kw):
        p = {k: FAKE for k in ("Q", "K", "V", "O", "L")}
        p.update(kw)
        return L.attn_mat_fwd(p["Q"], p["K"], p["V"], p["O"], p["L"], P, pb, 1, 1, n, 64, 0.125, 0, 0,
                              None)

    def bwd(P=FAKE, pb=P_OK, wsb=1 << 30, **kw):
        p = {k: FAKE for k in ("Q", "K", "V", "O", "dO", "dQ", "dK", "dV", "ws")}
        p.update(kw)
        return L.attn_mat_bwd(p["Q"], p["K"], p["V"], p["O"], p["dO"], P, pb, p["dQ"], p["dK"],
                              p["dV"], p["ws"], wsb, 1, 1, 8, 64, 0.125, 1, 0, None)

    def fb(P=FAKE, pb=P_OK, wsb=1 << 30, **kw):
        p = {k: FAKE for k in ("Q", "K", "V", "dO", "O", "L", "dQ", "dK", "dV", "ws")}
        p.update(kw)
        return L.attn_mat_fwd_bwd(p["Q"], p["K"], p["V"], p["dO"], p["O"], p["L"], P, pb, p["dQ"],
                                  p["dK"], p["dV"], p["ws"], wsb, 1, 1, 8, 64, 0.125, 0, 1, None)

    # fwd and bwd above are bfloat16 (P needs 8 * 128 * 2 bytes), fb float32
    for call, names, need in ((fwd, ("Q", "K", "V", "O", "L"), 8 * 128 * 2),
                              (bwd, ("Q", "K", "V", "O", "dO", "dQ", "dK", "dV", "ws"), 8 * 128 * 2),
                              (fb, ("Q", "K", "V", "dO", "O", "L", "dQ", "dK", "dV", "ws"), 8 * 128 * 4)):
        assert call(P=None) == -1
        assert call(P=MIS) == -4
        for name in names:
            assert call(**{name: None}) == -1, (call.__name__, name)
        assert call(pb=need - 1) == -5
    assert bwd(wsb=1) == -5
    assert fb(wsb=1) == -5
    assert fwd(n=(1 << 20) + 1) == -2


def test_binding_rejects_cpu_tensors():
    import torch
    import paper_2609_33916_amd as pkg
    x = torch.zeros(1, 1, 8, 32)
    with pytest.raises(ValueError):
        pkg.attn_fwd(x, x, x)


def test_library_source_never_allocates():
    """No device allocation anywhere in the library: all buffers are the
    caller's (the naive path's n x n P included), so the fused path can hold
    nothing of size n x n."""
    csrc = os.path.join(ROOT, "paper_2609_33916_amd", "csrc")
    for fn in os.listdir(csrc):
        text = open(os.path.join(csrc, fn)).read()
        for call in ("hipMalloc", "hipFree", "hipMallocAsync", "hipExtMalloc", "malloc("):
            assert call not in text, (fn, call)


def test_library_imports_no_allocator(L):
    """The built library links no device or host allocation routine of the
    HIP runtime, so nothing it runs can obtain an n x n buffer by itself."""
    import paper_2609_33916_amd as pkg
    import shutil
    import subprocess
    nm = shutil.which("nm")
    if nm is None:
        pytest.skip("nm not available")
    out = subprocess.run([nm, "-D", "--undefined-only", pkg.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    undefined = [line.split()[-1].split("@")[0] for line in out.splitlines() if line.strip()]
    assert "hipLaunchKernel" in undefined  # the listing is the library's imports
    banned = [s for s in undefined
              if re.match(r"hip(Ext)?(Malloc|Free|MemAlloc|MallocAsync|MallocManaged|HostMalloc|"
                          r"MallocPitch|Malloc3D|MallocArray|MemPool)", s)]
    assert banned == [], banned


def test_noalloc_size_limit_checked_on_the_host(L):
    """attn_fwd_bwd_noalloc rejects B * H * n beyond its fixed scratch (and
    the usual bad arguments) before any HIP call."""
    rows = L.attn_noalloc_max_rows()
    assert rows == (16 << 20) // 8
    call = lambda **kw: L.attn_fwd_bwd_noalloc(*(kw.get(k, FAKE) for k in
                                                 ("Q", "K", "V", "dO", "O", "L", "dQ", "dK", "dV")),
                                               kw.get("B", 1), kw.get("H", 1), kw.get("n", 8), kw.get("d", 64),
                                               0.125, 0, 0, None)
    assert call(n=rows + 1) == -8
    assert call(B=2, H=2, n=rows // 4 + 1) == -8
    assert call(Q=None) == -1
    assert call(dV=None) == -1
    assert call(d=48) == -3
    assert call(n=0) == -2
