"""CPU checks of the C ABI: the library loads, exports every function the
header declares, and its host-side logic (constants, the scale-bit rule, size
helpers, synchronous argument checks) behaves as documented.  Nothing here
launches a kernel."""
import ctypes
import subprocess

import pytest

import oracle
import paper_2609_09095_amd as oz


@pytest.fixture(scope="module", autouse=True)
def built_library():
    import os
    if not os.path.exists(oz.library_path()):
        from paper_2609_09095_amd import build
        build.build()
    oz.lib()


def test_header_symbols_are_exported():
    declared = oz.exported_symbols()
    assert "ozaki25_dgemm" in declared and "ozaki25_deconstruct" in declared
    assert "ozaki25_residue_gemm" in declared and "ozaki25_reconstruct" in declared
    out = subprocess.run(["nm", "-D", "--defined-only", oz.library_path()], capture_output=True,
                         text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    missing = [s for s in declared if s not in exported]
    assert not missing, missing
    for s in declared:
        getattr(oz.lib(), s)


def test_constants():
    assert oz.ozaki25_num_moduli() == 12
    assert oz.ozaki25_num_planes() == 30
    assert [oz.ozaki25_modulus(i) for i in range(12)] == oracle.moduli()
    assert oz.ozaki25_modulus(12) == -1 and oz.ozaki25_modulus(-1) == -1
    assert oz.ozaki25_num_moduli(7) == -1
    assert oz.ozaki25_status_string(0) == "success"
    assert "invalid" in oz.ozaki25_status_string(1)
    assert oz.ozaki25_status_string(99) == "unknown status"


def test_constants_all_byte_set():
    assert oz.ozaki25_num_moduli(oz.A15) == 15 == oz.NUM_MODULI_A15
    assert oz.ozaki25_num_planes(oz.A15) == 15
    assert [oz.ozaki25_modulus(i, oz.A15) for i in range(15)] == oracle.moduli(1)
    assert oz.ozaki25_modulus(15, oz.A15) == -1
    assert oz.ozaki25_num_moduli(2) == -1


@pytest.mark.parametrize("k", [1, 2, 63, 64, 65, 100, 255, 256, 1024, 4096, 7937, 8192, 4194304])
def test_scale_bits_matches_oracle(k):
    assert oz.ozaki25_scale_bits(k) == oracle.scale_bits(k)
    assert oz.ozaki25_scale_bits(k, oz.A15) == oracle.scale_bits(k, 1)


def test_scale_bits_invalid():
    assert oz.ozaki25_scale_bits(0) == -1
    assert oz.ozaki25_scale_bits(-5) == -1
    assert oz.ozaki25_scale_bits(64, 3) == -1


def test_size_helpers():
    assert oz.ozaki25_k_pad(0) == 0
    assert oz.ozaki25_k_pad(1) == 128 and oz.ozaki25_k_pad(128) == 128 and oz.ozaki25_k_pad(129) == 256
    assert oz.ozaki25_planes_bytes(10, 70) == 30 * 10 * 128
    assert oz.ozaki25_planes_bytes(10, 130) == 30 * 10 * 256
    assert oz.ozaki25_planes_bytes(-1, 70) == 0
    ws = oz.ozaki25_dgemm_workspace_size(100, 50, 70)
    assert ws >= 30 * 100 * 128 + 30 * 50 * 128 + 4 * 150 + 12 * 100 * 50 * 2
    assert ws % 256 == 0
    def up(x):
        return (x + 255) // 256 * 256
    # one tile per modulus, k = 70: a single k-split, just the residue products
    assert oz.ozaki25_dgemm_planes_workspace_size(100, 50, 70) == up(12 * 100 * 50 * 2)
    assert oz.ozaki25_dgemm_planes_workspace_size(100, 50, 70, oz.A15) == up(15 * 100 * 50)
    # 256 x 256 x 8192: 12 tiles split 16 ways (192 blocks: one round on 256 CUs)
    assert oz.ozaki25_dgemm_planes_workspace_size(256, 256, 8192) == up(12 * 256 * 256 * 2) * 17
    # 15 tiles: 16 ways for the int8 kernel (at least 4 stages per split)
    assert oz.ozaki25_dgemm_planes_workspace_size(256, 256, 8192, oz.A15) == up(15 * 256 * 256) * 17
    # 1024 x 1024 x 8192, int8: 240 tiles already fill one round
    assert oz.ozaki25_dgemm_planes_workspace_size(1024, 1024, 8192, oz.A15) == up(15 * 1024 * 1024)
    # enough tiles: no split
    assert oz.ozaki25_dgemm_planes_workspace_size(8192, 8192, 8192) == up(12 * 8192 * 8192 * 2)
    assert oz.ozaki25_dgemm_planes_workspace_size(100, 50, 70, 3) == 0
    # all-byte set: 15 int8 planes per operand, int8 residue products
    assert oz.ozaki25_planes_bytes(10, 70, oz.A15) == 15 * 10 * 128
    wa = oz.ozaki25_dgemm_workspace_size(100, 50, 70, oz.A15)
    assert 15 * 150 * 128 + 4 * 150 + 15 * 100 * 50 <= wa < ws and wa % 256 == 0


def _v(x):
    return ctypes.c_void_p(x)


def test_argument_errors_are_synchronous():
    L = oz.lib()
    fake = _v(0x100000)   # never dereferenced: every call below fails its checks first
    null = _v(0)
    # deconstruct: bad side, negative sizes, ldx too small, null pointers, bad set, k too large
    assert L.ozaki25_deconstruct(2, 4, 4, fake, 4, 0, 0, fake, fake, null) == oz.ERR_INVALID_VALUE
    assert L.ozaki25_deconstruct(0, -1, 4, fake, 4, 0, 0, fake, fake, null) == oz.ERR_INVALID_VALUE
    assert L.ozaki25_deconstruct(0, 4, 8, fake, 4, 0, 0, fake, fake, null) == oz.ERR_INVALID_VALUE
    assert L.ozaki25_deconstruct(1, 8, 4, fake, 4, 0, 0, fake, fake, null) == oz.ERR_INVALID_VALUE
    assert L.ozaki25_deconstruct(0, 4, 4, null, 4, 0, 0, fake, fake, null) == oz.ERR_INVALID_VALUE
    assert L.ozaki25_deconstruct(0, 4, 4, fake, 4, 5, 0, fake, fake, null) == oz.ERR_INVALID_VALUE
    assert L.ozaki25_deconstruct(0, 4, 4, fake, 4, 0, 2, fake, fake, null) == oz.ERR_INVALID_VALUE
    assert L.ozaki25_deconstruct(0, 4, oz.MAX_K + 1, fake, oz.MAX_K + 1, 0, 0, fake, fake, null) == oz.ERR_UNSUPPORTED
    assert L.ozaki25_deconstruct(0, 4, 4, fake, 4, 0, 0, _v(0x100001), fake, null) == oz.ERR_INVALID_VALUE
    # empty work is a successful no-op
    assert L.ozaki25_deconstruct(0, 0, 4, null, 4, 0, 0, null, null, null) == oz.SUCCESS
    assert L.ozaki25_deconstruct(0, 4, 0, null, 4, 0, 0, null, null, null) == oz.SUCCESS
    # residue gemm
    assert L.ozaki25_residue_gemm(4, 4, 4, null, fake, 0, fake, null) == oz.ERR_INVALID_VALUE
    assert L.ozaki25_residue_gemm(4, 4, 4, fake, fake, 0, null, null) == oz.ERR_INVALID_VALUE
    assert L.ozaki25_residue_gemm(0, 4, 4, null, null, 0, null, null) == oz.SUCCESS
    assert L.ozaki25_residue_gemm(4, 4, oz.MAX_K + 1, fake, fake, 0, fake, null) == oz.ERR_UNSUPPORTED
    assert L.ozaki25_residue_gemm(4, oz.MAX_N + 1, 4, fake, fake, 0, fake, null) == oz.ERR_UNSUPPORTED
    # reconstruct
    assert L.ozaki25_reconstruct(4, 4, fake, fake, fake, 0, fake, 3, 0, null) == oz.ERR_INVALID_VALUE
    assert L.ozaki25_reconstruct(4, 4, null, fake, fake, 0, fake, 4, 0, null) == oz.ERR_INVALID_VALUE
    assert L.ozaki25_reconstruct(4, 0, null, null, null, 0, null, 0, 0, null) == oz.SUCCESS
    # dgemm: leading dimensions, aliasing, null pointers
    f = L.ozaki25_dgemm_ex
    assert f(4, 4, 4, fake, 3, fake, 4, _v(0x200000), 4, 0, 0, 0, null, 0, null, null) == oz.ERR_INVALID_VALUE
    assert f(4, 4, 4, fake, 4, fake, 3, _v(0x200000), 4, 0, 0, 0, null, 0, null, null) == oz.ERR_INVALID_VALUE
    assert f(4, 4, 4, fake, 4, _v(0x300000), 4, _v(0x200000), 3, 0, 0, 0, null, 0, null, null) == oz.ERR_INVALID_VALUE
    assert f(4, 4, 4, fake, 4, _v(0x300000), 4, fake, 4, 0, 0, 0, null, 0, null, null) == oz.ERR_INVALID_VALUE
    assert f(4, 4, 4, null, 4, _v(0x300000), 4, _v(0x200000), 4, 0, 0, 0, null, 0, null, null) == oz.ERR_INVALID_VALUE
    assert f(4, 4, 4, fake, 4, _v(0x300000), 4, _v(0x200000), 4, 2, 0, 0, null, 0, null, null) == oz.ERR_INVALID_VALUE
    assert f(4, 4, 4, fake, 4, _v(0x300000), 4, _v(0x200000), 4, 0, 2, 0, null, 0, null, null) == oz.ERR_INVALID_VALUE
    assert f(0, 4, 4, null, 4, null, 4, null, 4, 0, 0, 0, null, 0, null, null) == oz.SUCCESS
    assert f(4, oz.MAX_N + 1, 4, fake, 4, _v(0x300000), oz.MAX_N + 1, _v(0x200000), oz.MAX_N + 1, 0, 0, 0, null, 0, null, null) == oz.ERR_UNSUPPORTED
    # a caller workspace that is too small is refused before any launch
    assert f(4, 4, 4, fake, 4, _v(0x300000), 4, _v(0x200000), 4, 0, 0, 0, _v(0x400000), 16, null, null) == oz.ERR_WORKSPACE
    # dgemm from stored planes
    g = L.ozaki25_dgemm_planes
    pa, ea, pb, eb, c = _v(0x100000), _v(0x200000), _v(0x300000), _v(0x400000), _v(0x500000)
    assert g(4, 4, 4, pa, ea, pb, eb, c, 3, 0, 0, null, 0, null) == oz.ERR_INVALID_VALUE     # ldc < n
    assert g(4, 4, 4, null, ea, pb, eb, c, 4, 0, 0, null, 0, null) == oz.ERR_INVALID_VALUE   # no planes
    assert g(4, 4, 4, pa, null, pb, eb, c, 4, 0, 0, null, 0, null) == oz.ERR_INVALID_VALUE   # no exponents
    assert g(4, 4, 4, pa, ea, pb, eb, c, 4, 2, 0, null, 0, null) == oz.ERR_INVALID_VALUE     # bad set
    assert g(4, 4, 4, _v(0x100008), ea, pb, eb, c, 4, 0, 0, null, 0, null) == oz.ERR_INVALID_VALUE
    assert g(4, 4, oz.MAX_K + 1, pa, ea, pb, eb, c, 4, 0, 0, null, 0, null) == oz.ERR_UNSUPPORTED
    assert g(0, 4, 4, null, null, null, null, null, 4, 0, 0, null, 0, null) == oz.SUCCESS
    assert g(4, 4, 4, pa, ea, pb, eb, c, 4, 0, 0, _v(0x600000), 8, null) == oz.ERR_WORKSPACE
    # the dgemm workspace grows by the split-k partials for few output tiles
    assert (oz.ozaki25_dgemm_workspace_size(256, 256, 8192)
            >= oz.ozaki25_dgemm_planes_workspace_size(256, 256, 8192) + 2 * 30 * 256 * 8192)


def test_binding_fails_loudly_without_library(tmp_path, monkeypatch):
    monkeypatch.setattr(oz, "_LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(oz, "_lib", None)
    with pytest.raises(ImportError):
        oz.lib()


def test_noalloc_limit_is_checked_on_the_host():
    """ozaki25_dgemm_noalloc refuses a product whose workspace exceeds its
    static array before any HIP call (so this runs without a GPU), and the
    header's constant matches the binding's."""
    L = oz.lib()
    assert oz.NOALLOC_SCRATCH_BYTES == 128 << 20
    fake = ctypes.c_void_p(1 << 20)
    m = n = k = 2048
    assert oz.ozaki25_dgemm_workspace_size(m, n, k) > oz.NOALLOC_SCRATCH_BYTES
    st = L.ozaki25_dgemm_noalloc(m, n, k, fake, k, fake, n, fake, n, oz.S12, oz.RN, 0, None)
    assert st == oz.ERR_WORKSPACE
    assert L.ozaki25_dgemm_noalloc(-1, n, k, fake, k, fake, n, fake, n, oz.S12, oz.RN, 0, None) == oz.ERR_INVALID_VALUE
    assert L.ozaki25_dgemm_noalloc(m, n, k, fake, k, fake, n, fake, n, 5, oz.RN, 0, None) == oz.ERR_INVALID_VALUE
    assert L.ozaki25_dgemm_noalloc(0, n, k, fake, k, fake, n, fake, n, oz.S12, oz.RN, 0, None) == oz.SUCCESS
    for s in (oz.S12, oz.A15):
        assert oz.ozaki25_dgemm_workspace_size(1024, 1024, 1024, s) <= oz.NOALLOC_SCRATCH_BYTES
