"""Host-side checks of the C ABI: the library loads, exports every entry point the
header declares, sizes the packed weights as documented, and rejects invalid
arguments with the documented status before launching anything (so these run
without a GPU: no call here reaches a kernel launch)."""
import ctypes
import os
import re

import pytest

import __graft_entry__ as graft

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "flashnorm.h")


@pytest.fixture(scope="module")
def fnlib():
    graft.ensure_built()
    from paper_2407_09577_amd import flashnorm
    return flashnorm


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\*?\s+\**([a-z_0-9]+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_header_declares_the_boundary():
    names = _declared_functions()
    for required in ("fold_weights", "flashnorm_linear", "flashnorm_glu", "flashnorm_layernorm_linear"):
        assert required in names
    assert len(names) >= 13


def test_library_exports_every_declared_symbol(fnlib):
    lib = ctypes.CDLL(fnlib.LIB_PATH)
    missing = [n for n in _declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings(fnlib):
    lib = fnlib.lib()
    for code, name in fnlib.STATUS.items():
        assert lib.flashnorm_status_string(code).decode().startswith(name)
    assert lib.flashnorm_status_string(12345).decode() == "unknown fn_status"


def test_fold_weights_size(fnlib):
    f = fnlib.fold_weights_size
    # bf16: rows padded to 64, columns to 16; GLU: 2 * round_up(F, 16) columns
    assert f(576, 1536, 0, 1) == 576 * 1536 * 2
    assert f(4096, 22016, 1, 1) == 4096 * 22016 * 2
    assert f(576, 576, 0, 0) == 576 * 576 * 4
    assert f(8, 3, 0, 1) == 64 * 16 * 2
    assert f(72, 2 * 9, 1, 1) == 128 * 32 * 2
    assert f(0, 16, 0, 1) == 0 and f(16, 0, 0, 1) == 0
    assert f(16, 7, 1, 1) == 0          # GLU needs an even column count
    assert f(16, 16, 2, 1) == 0          # unknown layout
    assert f(16, 16, 0, 7) == 0          # unknown dtype
    # packed buffers of 2^31 bytes or more are beyond the kernels' 32-bit offsets
    assert f(1 << 15, (1 << 15) - 16, 0, 1) == (1 << 15) * ((1 << 15) - 16) * 2
    assert f(1 << 15, 1 << 15, 0, 1) == 0
    assert f(1 << 15, 1 << 14, 0, 0) == 0


# Fake but aligned, non-null device addresses: validation never dereferences them.
A, W, Y, X = 0x100000, 0x200000, 0x300000, 0x400000


def _lin(lib, a=A, M=4, K=64, lda=64, adt=1, ws=W, N=32, eps=1e-6, y=Y, ldy=32, ydt=1, path=0):
    return lib.flashnorm_linear_ex(a, M, K, lda, adt, ws, N, eps, None, y, ldy, ydt, None, path, None)


def test_linear_validation(fnlib):
    lib = fnlib.lib()
    assert _lin(lib, M=-1) == -2
    assert _lin(lib, K=0) == -2
    assert _lin(lib, N=0) == -2
    assert _lin(lib, lda=32) == -2                 # lda < K
    assert _lin(lib, K=60, lda=64) == -2           # bf16 K % 8
    assert _lin(lib, ldy=16) == -2                 # ldy < N
    assert _lin(lib, a=0) == -1
    assert _lin(lib, ws=0) == -1
    assert _lin(lib, y=0) == -1
    assert _lin(lib, a=A + 8) == -4                # 16-byte alignment
    assert _lin(lib, lda=68, K=64) == -4           # row alignment (bf16: ld % 8)
    assert _lin(lib, adt=5) == -3
    assert _lin(lib, ydt=0) == -3                  # output dtype must match
    assert _lin(lib, eps=-1.0) == -6
    assert _lin(lib, eps=float("nan")) == -6
    assert _lin(lib, eps=float("inf")) == -6
    assert _lin(lib, path=7) == -6
    assert _lin(lib, M=17, path=2) == -5           # decode path takes M <= 16
    assert _lin(lib, adt=0, ydt=0, path=2) == -5   # decode path is bf16 only
    assert _lin(lib, y=A + 64) == -8               # output overlaps the activations
    assert _lin(lib, lda=1 << 22, K=64) == -9
    assert _lin(lib, K=1 << 15, lda=1 << 15, N=1 << 15, ldy=1 << 15) == -9   # 2 GiB packed weight
    # M == 0 is a no-op that never touches the device, even with null tensors
    assert _lin(lib, M=0, a=0, y=0) == 0


def test_glu_and_layernorm_validation(fnlib):
    lib = fnlib.lib()
    glu = lambda **kw: lib.flashnorm_glu_ex(kw.get("a", A), kw.get("M", 4), 64, 64, 1, kw.get("ws", W),
                                            kw.get("F", 16), 1e-6, Y, kw.get("ldo", 16), 1, 0, None)
    assert glu(F=0) == -2
    assert glu(ws=0) == -1
    assert glu(ldo=8) == -2
    ln = lambda **kw: lib.flashnorm_layernorm_linear_ex(A, 4, 64, 64, 1, W, kw.get("colsum", X), None, 32,
                                                        kw.get("eps", 1e-5), Y, 32, 1, 0, None)
    assert ln(colsum=0) == -1
    assert ln(eps=-1e-3) == -6


def test_fold_validation(fnlib):
    lib = fnlib.lib()
    f = lambda **kw: lib.fold_weights(kw.get("W", A), kw.get("sk", 32), kw.get("sn", 1), kw.get("wdt", 1), kw.get("g", X),
                                      kw.get("beta", None), kw.get("K", 64), kw.get("N", 32),
                                      kw.get("layout", 0), kw.get("ws", W), kw.get("wsdt", 1),
                                      kw.get("colsum", None), kw.get("cstar", None), None)
    assert f(W=0) == -1
    assert f(ws=0) == -1
    assert f(sk=-32) == -2                         # negative strides
    assert f(sn=-1) == -2
    assert f(N=31, layout=1) == -2
    assert f(sk=1 << 40) == -9                     # element offsets must stay below 2^62
    assert f(sn=1 << 31) == -9
    assert f(layout=3) == -6
    assert f(wdt=4) == -3
    assert f(cstar=X) == -1                        # c* needs beta
    assert f(layout=1, colsum=X) == -5             # LayerNorm extras: linear layout only
    assert f(ws=W + 4) == -4
    assert f(ws=A + 16) == -8                      # packed output overlaps W
    assert f(K=1 << 15, N=1 << 15, sk=1 << 15) == -9
    assert f(ws=A + 64 * 32 * 2 - 16) == -8        # overlaps the last element of the row-major view
    assert f(sk=1, sn=64, ws=A + 32 * 64 * 2 - 16) == -8   # and of the transposed view
    u = lambda **kw: lib.unpack_weights(kw.get("ws", W), 64, 32, 0, 1, kw.get("out", Y), kw.get("ldo", 32), None)
    assert u(ws=0) == -1
    assert u(ldo=8) == -2


def test_baseline_validation(fnlib):
    lib = fnlib.lib()
    b = lambda **kw: lib.baseline_rmsnorm_linear(A, 4, 64, 64, 1, kw.get("g", X), W, 32, 1e-6,
                                                 kw.get("xws", 0x500000), Y, 32, 0, None)
    assert b(g=0) == -1
    assert b(xws=0) == -1
    assert b(xws=A) == -8                          # workspace overlaps the activations
    assert lib.baseline_layernorm_linear(A, 4, 64, 64, 1, X, None, W, 32, 1e-5, 0x500000, Y, 32, 0, None) == -1


def test_vector_alignment_validation(fnlib):
    lib = fnlib.lib()
    assert lib.flashnorm_linear_ex(A, 4, 64, 64, 1, W, 32, 1e-6, X + 4, Y, 32, 1, None, 0, None) == -4
    assert lib.flashnorm_layernorm_linear_ex(A, 4, 64, 64, 1, W, X + 8, None, 32, 1e-5, Y, 32, 1, 0, None) == -4
    assert lib.flashnorm_layernorm_linear_ex(A, 4, 64, 64, 1, W, X, X + 4, 32, 1e-5, Y, 32, 1, 0, None) == -4


def test_epilogue_family_validation(fnlib):
    lib = fnlib.lib()
    ga = lambda **kw: lib.flashnorm_glu_act(A, kw.get("M", 4), 64, 64, 1, W, 16, 1e-6, kw.get("act", 0), Y, 16, 1,
                                            kw.get("inv", None), kw.get("path", 0), None)
    assert ga(act=7) == -6                          # unknown gate nonlinearity
    assert ga(act=3) == -1                          # deferred up scale: inv_rms must be given
    assert ga(act=1, inv=X) == -6                   # ReGLU / bilinear carry the whole scale
    assert ga(act=2, inv=X) == -6
    assert ga(act=0, path=1 | (3 << 8)) == -5       # forced tile: automatic configuration only
    assert ga(act=3, M=0) == 0                      # M == 0: no-op
    lr = lambda **kw: lib.flashnorm_linear_relu(A, 4, 64, 64, 1, W, 32, 1e-6, Y, 32, 1, kw.get("inv", X),
                                                kw.get("path", 0), None)
    assert lr(inv=0) == -1
    assert lr(path=2 | (1 << 8)) == -5
    rs = lambda **kw: lib.rowscale_linear(A, 4, 64, 64, 1, W, 32, kw.get("s", X), Y, 32, kw.get("ydt", 1), 0, None)
    assert rs(s=0) == -1
    assert rs(ydt=0) == -3


def test_unfolded_validation(fnlib):
    lib = fnlib.lib()
    lu = lambda **kw: lib.flashnorm_linear_unfolded(A, kw.get("M", 64), kw.get("K", 64), kw.get("K", 64), 1,
                                                    kw.get("g", X), W, 32, 1e-6, None, Y, 32, 1, None,
                                                    kw.get("path", 0), None)
    assert lu(g=0) == -1                            # run-time g must be given
    assert lu(g=X + 4) == -4
    assert lu(g=Y) == -8                            # g overlaps the output
    assert lu(path=1 | (2 << 8)) == -5              # forced tile: automatic configuration only
    assert lu(K=8136) == -5                         # bf16 tile path stages g in LDS: K <= 8128
    assert lu(M=0, g=0) == 0                        # M == 0: no-op
    gu = lambda **kw: lib.flashnorm_glu_unfolded(A, kw.get("M", 64), 8200, 8200, 1, kw.get("g", X), W, 16, 1e-6,
                                                 Y, 16, 1, kw.get("path", 0), None)
    assert gu(g=0) == -1
    assert gu(path=1) == -5


def test_qkv_rope_validation(fnlib):
    lib = fnlib.lib()
    T, S, Pz = 0x500000, 0x600000, 0x700000    # cos, sin tables and positions (never dereferenced)

    def qr(**kw):
        return lib.flashnorm_qkv_rope(A, kw.get("M", 4), 64, 64, kw.get("dt", 1), W, kw.get("Hq", 2), kw.get("Hkv", 1),
                                      kw.get("h", 8), 1e-6, kw.get("bias", None), kw.get("pos", Pz), kw.get("cos", T),
                                      kw.get("sin", S), kw.get("P", 16), kw.get("qs", 0.5), kw.get("y", Y), 32,
                                      kw.get("dt", 1), None, kw.get("path", 0), None)
    assert qr(h=6) == -2                            # head width a multiple of 4
    assert qr(h=0) == -2 and qr(Hq=0) == -2 and qr(Hkv=-1) == -2 and qr(P=0) == -2
    assert qr(qs=float("inf")) == -6
    assert qr(pos=0) == -1 and qr(cos=0) == -1 and qr(sin=0) == -1
    assert qr(cos=T + 8) == -4 and qr(pos=Pz + 4) == -4 and qr(bias=X + 4) == -4
    assert qr(y=T) == -8                            # output overlaps a table
    assert qr(path=1 | (2 << 8)) == -5              # automatic configuration only
    assert qr(M=0, pos=0) == 0                      # M == 0: no-op


def test_baseline_rope_validation(fnlib):
    lib = fnlib.lib()
    T, S, Pz = 0x500000, 0x600000, 0x700000

    def br(**kw):
        return lib.baseline_rope(kw.get("y", Y), kw.get("M", 4), kw.get("ld", 32), kw.get("dt", 1), 2, 1,
                                 kw.get("h", 8), kw.get("pos", Pz), T, S, 16, 0.5, None)
    assert br(h=2) == -2
    assert br(ld=16) == -2                          # ldy below the Q and K columns
    assert br(dt=5) == -3
    assert br(pos=0) == -1
    assert br(pos=Pz + 4) == -4
    assert br(y=T) == -8
    assert br(M=0, pos=0) == 0


def test_qkv_headnorm_validation(fnlib):
    lib = fnlib.lib()
    G1, G2, T, S, Pz = 0x500000, 0x510000, 0x600000, 0x610000, 0x700000

    def hn(**kw):
        return lib.flashnorm_qkv_headnorm(A, kw.get("M", 4), 64, 64, kw.get("dt", 1), W, 2, 1, kw.get("h", 8), 1e-6,
                                          kw.get("gq", G1), kw.get("gk", G2), kw.get("gv", None), kw.get("eh", 1e-6),
                                          kw.get("pos", Pz), kw.get("cos", T), kw.get("sin", S), 16, 0.5,
                                          kw.get("y", Y), kw.get("ldy", 32), kw.get("dt", 1), None, kw.get("path", 0),
                                          None)
    assert hn(h=12) == -2 and hn(h=4) == -2        # head width: a power of two from 8 to 256
    assert hn(dt=0, h=128, ldy=512) == -5           # fp32: heads up to 64 wide
    assert hn(eh=-1.0) == -6 and hn(eh=float("nan")) == -6
    assert hn(gq=0) == -1 and hn(gk=0) == -1
    assert hn(cos=0) == -1                          # positions need the tables
    assert hn(pos=0, cos=0, sin=0, y=G1) == -8      # no positions: no tables needed (stops at the alias check)
    assert hn(gv=G1 + 4) == -4
    assert hn(y=G1) == -8
    assert hn(path=1 | (3 << 8)) == -5
    assert hn(M=0, gq=0) == 0


def test_baseline_qkv_headnorm_validation(fnlib):
    lib = fnlib.lib()
    G1, G2, T, S, Pz = 0x500000, 0x510000, 0x600000, 0x610000, 0x700000

    def bh(**kw):
        return lib.baseline_qkv_headnorm(Y, kw.get("M", 4), kw.get("ld", 32), kw.get("dt", 1), 2, 1, kw.get("h", 8),
                                         kw.get("gq", G1), G2, None, 1e-6, kw.get("pos", Pz), T, S, 16, 0.5, None)
    assert bh(h=6) == -2 and bh(dt=0) == -5 and bh(dt=7) == -3
    assert bh(ld=16) == -2                          # ldy below the normalised columns
    assert bh(gq=0) == -1 and bh(pos=Pz + 4) == -4
    assert bh(M=0, gq=0) == 0


def test_mla_latent_validation(fnlib):
    lib = fnlib.lib()
    T, S, Pz, G = 0x500000, 0x600000, 0x700000, 0x800000   # tables, positions, g_lat (never dereferenced)

    def ml(**kw):
        return lib.flashnorm_mla_latent(A, kw.get("M", 4), 64, 64, kw.get("dt", 1), W, kw.get("L", 16),
                                        kw.get("R", 8), kw.get("g", G), kw.get("el", 1e-6), 1e-6, kw.get("pos", Pz),
                                        kw.get("cos", T), kw.get("sin", S), kw.get("P", 16), kw.get("y", Y), 32,
                                        kw.get("dt", 1), kw.get("inv", X), kw.get("path", 0), None)
    assert ml(L=12) == -2 and ml(L=0) == -2 and ml(L=2056) == -2   # latent: multiple of 8, <= 2048
    assert ml(R=4) == -2 and ml(R=-8) == -2 and ml(R=520) == -2    # rotary: multiple of 8, <= 512
    assert ml(P=0) == -2
    assert ml(el=-1.0) == -6 and ml(el=float("nan")) == -6
    assert ml(g=0) == -1 and ml(pos=0) == -1 and ml(cos=0) == -1 and ml(inv=0) == -1
    assert ml(g=G + 4) == -4 and ml(cos=T + 8) == -4 and ml(pos=Pz + 4) == -4
    assert ml(y=T) == -8                            # output overlaps a table
    assert ml(y=G) == -8                            # output overlaps g_lat
    assert ml(dt=7) == -3
    assert ml(M=0, g=0, pos=0) == 0                 # M == 0: no-op
    assert ml(R=0, P=0, M=0) == 0 and ml(R=8, P=0, M=0) == -2   # the tables matter only with a rotary part
    bl = lambda **kw: lib.baseline_mla_latent(kw.get("y", Y), kw.get("M", 4), 32, kw.get("dt", 1), kw.get("L", 16),
                                              kw.get("R", 8), kw.get("g", G), 1e-6, kw.get("pos", Pz), T, S,
                                              kw.get("P", 16), None)
    assert bl(L=10) == -2 and bl(R=6) == -2 and bl(L=32, R=8) == -2   # L + R wider than ldy
    assert bl(g=0) == -1 and bl(pos=0) == -1
    assert bl(y=Y + 4) == -4
    assert bl(dt=5) == -3
    assert bl(M=0) == 0


# ----------------------------------------------------------- the Python binding's own guards
# The C ABI cannot see tensor sizes or devices, so the binding refuses, before any call,
# arguments that would make a kernel read or write outside an allocation.  These run on
# host tensors: the size checks come before the device check, so each rejection is the
# one named.
def _bf16(*shape):
    import torch
    return torch.zeros(*shape, dtype=torch.bfloat16)


def test_binding_rejects_short_packed_weight(fnlib):
    M, K, N = 4, 64, 32
    need = fnlib.fold_weights_size(K, N, fnlib.FN_LAYOUT_LINEAR, fnlib.FN_BF16)
    import torch
    short = torch.zeros(need - 16, dtype=torch.uint8)
    with pytest.raises(ValueError, match="packed weight holds"):
        fnlib.flashnorm_linear(_bf16(M, K), short, N, 1e-6)
    # a weight folded for fewer columns, reused for more
    with pytest.raises(ValueError, match="packed weight holds"):
        fnlib.flashnorm_linear(_bf16(M, K), torch.zeros(need, dtype=torch.uint8), 2 * N, 1e-6)
    glu_need = fnlib.fold_weights_size(K, 2 * N, fnlib.FN_LAYOUT_GLU, fnlib.FN_BF16)
    with pytest.raises(ValueError, match="packed weight holds"):
        fnlib.flashnorm_glu(_bf16(M, K), torch.zeros(glu_need - 1024, dtype=torch.uint8), N, 1e-6)
    with pytest.raises(ValueError, match="packed weight holds"):
        fnlib.flashnorm_layernorm_linear(_bf16(M, 2 * K), torch.zeros(need, dtype=torch.uint8),
                                         torch.zeros(N), None, N, 1e-6)
    with pytest.raises(ValueError, match="packed weight holds"):
        fnlib.baseline_rmsnorm_linear(_bf16(M, K), torch.ones(K), short, N, 1e-6)


def test_binding_rejects_wrong_output_and_workspace(fnlib):
    import torch
    M, K, N = 4, 64, 32
    Ws = torch.zeros(fnlib.fold_weights_size(K, N, fnlib.FN_LAYOUT_LINEAR, fnlib.FN_BF16), dtype=torch.uint8)
    with pytest.raises(ValueError, match="output of shape"):
        fnlib.flashnorm_linear(_bf16(M, K), Ws, N, 1e-6, out=_bf16(M - 1, N))
    with pytest.raises(ValueError, match="workspace"):
        fnlib.baseline_rmsnorm_linear(_bf16(M, K), torch.ones(K), Ws, N, 1e-6, x_ws=_bf16(M - 1, K))
    with pytest.raises(ValueError, match="output of shape"):
        fnlib.baseline_rope(_bf16(M, 100), 1, 1, 32, torch.zeros(M, dtype=torch.int32), torch.zeros(8, 16),
                            torch.zeros(8, 16), 1.0)
    with pytest.raises(ValueError, match="cos_tab"):
        fnlib.baseline_rope(_bf16(M, 96), 1, 1, 32, torch.zeros(M, dtype=torch.int32), torch.zeros(8, 8),
                            torch.zeros(8, 8), 1.0)


def test_binding_rejects_host_tensors(fnlib):
    import torch
    M, K, N = 4, 64, 32
    Ws = torch.zeros(fnlib.fold_weights_size(K, N, fnlib.FN_LAYOUT_LINEAR, fnlib.FN_BF16), dtype=torch.uint8)
    with pytest.raises(ValueError, match="GPU tensor"):
        fnlib.flashnorm_linear(_bf16(M, K), Ws, N, 1e-6)
    with pytest.raises(ValueError, match="GPU tensor"):
        fnlib.fold_weights(_bf16(K, N), torch.ones(K))
    with pytest.raises(ValueError, match="GPU tensor"):
        fnlib.flashnorm_layernorm_linear(_bf16(M, K), Ws, torch.zeros(N), None, N, 1e-6)


def test_noalloc_baseline_validation(fnlib):
    # The static-workspace entry point rejects activations larger than its array before
    # touching the device, and M == 0 is a no-op (no device call at all).
    lib = fnlib.lib()
    f = lambda **kw: lib.baseline_rmsnorm_linear_noalloc(A, kw.get("M", 4), kw.get("K", 64), kw.get("K", 64),
                                                         kw.get("dt", 1), X, W, 32, 1e-6, Y, 32, 0, None)
    cap = fnlib.FN_NOALLOC_SCRATCH_BYTES
    assert f(M=cap // (2 * 4096) + 1, K=4096) == -9      # one row more than fits (bf16)
    assert f(M=cap // (4 * 4096) + 1, K=4096, dt=0) == -9  # fp32
    assert f(M=-1) == -2
    assert f(dt=7) == -3
    assert f(M=0) == 0


def test_binding_pads_the_outputs_it_allocates(fnlib):
    # Outputs the caller does not pass are allocated with a 16-byte row pitch (the pitch the
    # kernels' vector stores need), so any output width works; widths that are already a
    # multiple of 16 bytes get a plain contiguous tensor.
    import torch
    for dtype, per in ((torch.bfloat16, 8), (torch.float32, 4)):
        like = torch.zeros(1, dtype=dtype)
        for n in (1, per - 1, per, 45, 333, 1024):
            y = fnlib._new_out(3, n, like)
            assert tuple(y.shape) == (3, n) and y.dtype == dtype and y.stride(1) == 1
            assert y.stride(0) % per == 0 and y.stride(0) - n < per
            assert y.is_contiguous() == (n % per == 0)
