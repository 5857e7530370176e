"""Host-side checks of the C ABI library (no GPU): it loads, exports everything include/tvq.h
declares, and its host-only helpers agree with the independently written oracle."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def tvq():
    import paper_2603_27467_amd as tvq
    tvq.load_library()
    return tvq


def _declared_symbols():
    src = open(os.path.join(ROOT, "include", "tvq.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tvq_[a-z_0-9]+)\s*\(", src)))


def test_library_exports_every_declared_symbol(tvq):
    syms = _declared_symbols()
    assert {"tvq_create", "tvq_destroy", "tvq_cache_layout", "tvq_encode", "tvq_decode",
            "tvq_bits_per_element", "tvq_status_string"} <= set(syms)
    lib = ctypes.CDLL(tvq.library_path())
    missing = [s for s in syms if not hasattr(lib, s)]
    assert not missing, missing
    header = open(os.path.join(ROOT, "include", "tvq.h")).read()
    assert tvq.tvq_abi_version() == int(re.search(r"#define TVQ_ABI_VERSION (\d+)", header).group(1))


def test_status_strings(tvq):
    assert tvq.tvq_status_string(0) == "ok"
    assert "invalid" in tvq.tvq_status_string(-1)
    assert tvq.tvq_status_string(-99) == "unknown status"


@pytest.mark.parametrize("seed", [0, 1, 102, 2**63 + 5])
def test_signs_agree_with_oracle(tvq, orc, seed):
    """Both sides implement SplitMix64 from its published definition; they must agree."""
    for layer in (0, 1, 31):
        for d in (64, 128):
            assert np.array_equal(tvq.tvq_make_signs(seed, layer, d), orc.signs(seed, layer, d))


def test_trig_table_agrees_with_oracle(tvq, orc):
    """The reconstruction lookup (section 3.1) of every codebook size 2..4096, bit for bit."""
    for n in range(2, 4097):
        c1, s1 = tvq.tvq_make_trig_table(n)
        c2, s2 = orc.trig_table(n)
        assert np.array_equal(c1.view(np.uint32), c2.view(np.uint32)), n
        assert np.array_equal(s1.view(np.uint32), s2.view(np.uint32)), n


def test_decode_table_agrees_with_oracle(tvq, orc):
    """The table the decode kernels read (1/sqrt(d) folded in), bit for bit, d = 64 and 128."""
    for d in (64, 128):
        for n in list(range(2, 300)) + [384, 512, 1000, 2048, 4095, 4096]:
            c1, s1 = tvq.tvq_make_decode_table(n, d)
            c2, s2 = orc.decode_table(n, d)
            assert np.array_equal(c1.view(np.uint32), c2.view(np.uint32)), (n, d)
            assert np.array_equal(s1.view(np.uint32), s2.view(np.uint32)), (n, d)


def _cfg(tvq, table, L, H, d, seed=0, shared=0, signs=None, packing=0):
    arr = (tvq.tvq_layer_cfg * max(len(table), 1))()
    for i, t in enumerate(table):
        arr[i] = tvq.tvq_layer_cfg(*t)
    sp = None
    if signs is not None:
        signs = np.ascontiguousarray(signs, np.int8)
        sp = signs.ctypes.data_as(ctypes.POINTER(ctypes.c_int8))
    cfg = tvq.tvq_config(L, H, d, shared, seed, arr, sp, packing)
    cfg._keep = (arr, signs)
    return cfg


def _random_table(rng, L):
    out = []
    for _ in range(L):
        row = []
        for _kind in range(2):
            n = int(rng.choice([2, 3, 8, 32, 48, 56, 64, 100, 128, 256, 4096]))
            mode = int(rng.integers(0, 3))
            bits = 32 if mode == 0 else int(rng.integers(1, 17))
            row.append((n, bits, mode))
        (nk, bk, mk), (nv, bv, mv) = row
        out.append((nk, nv, bk, bv, mk, mv))
    return out


@pytest.mark.parametrize("seed", range(6))
def test_layout_agrees_with_oracle(tvq, orc, seed):
    """Layouts of random tables, with and without group packing (odd seeds)."""
    rng = np.random.default_rng(seed)
    packing = seed % 2
    L = int(rng.integers(1, 9))
    H = int(rng.integers(1, 9))
    d = int(rng.choice([64, 128]))
    B = int(rng.integers(1, 4))
    T = int(rng.integers(1, 300))
    table = _random_table(rng, L)
    lay = tvq.tvq_layout_for_config(_cfg(tvq, table, L, H, d, packing=packing), B, T)
    kinds = []
    for (nk, nv, bk, bv, mk, mv) in table:
        kinds += [orc.Kind(nk, mk, bk), orc.Kind(nv, mv, bv)]
    oc = orc.Codec(L, H, d, kinds, np.ones((L, d), np.int8), packing=packing)
    total, off = oc.layout(B, T)
    assert lay.total_bytes == total
    assert lay.batch == B and lay.capacity_tokens == T
    for l in range(L):
        for k in range(2):
            assert list(lay.off[l][k]) == list(off[l, k])
            assert list(lay.rec_bytes[l][k]) == oc.record_bytes(l, k)


def _expand(spec):
    out = []
    for g in spec.split():
        v, c = g.split("x")
        out += [int(v)] * int(c)
    return out


def test_bits_per_element_matches_paper_rates(tvq):
    """tvq_bits_per_element_config, accounting 0, against the rates printed in the paper."""
    rows = []
    for line in open(os.path.join(ROOT, "tests", "golden", "paper_rates.txt")):
        if line.strip() and not line.startswith("#"):
            rows.append([x.strip() for x in line.split("|")])
    checked = 0
    for label, nk, nv, bk, bv, d, printed, what in rows:
        nk, nv = _expand(nk), _expand(nv)
        L, bk, bv, d, printed = len(nk), int(bk), int(bv), int(d), float(printed)
        if what == "angle":
            # angle-only rates: fp32 norms add exactly 16 bits (section 3.1 "Rate accounting")
            table = [(a, b, 32, 32, 0, 0) for a, b in zip(nk, nv)]
            got = tvq.tvq_bits_per_element_config(_cfg(tvq, table, L, 8, d), 0) - 16.0
        elif what == "total":
            table = [(a, b, bk, bv, 1, 2) for a, b in zip(nk, nv)]
            got = tvq.tvq_bits_per_element_config(_cfg(tvq, table, L, 8, d), 0)
        else:
            continue
        assert abs(got - printed) <= 0.005 + 1e-9, (label, got, printed)
        checked += 1
    assert checked >= 20


def test_bits_per_element_storage(tvq):
    """Accounting 1 is the real layout: Mistral-shaped K8 linear / V4 log at n=64 stores
    120 + 88 bytes per (K, V) vector pair of d=128, i.e. 6.5 bits per element."""
    table = [(64, 64, 8, 4, 1, 2)] * 32
    cfg = _cfg(tvq, table, 32, 8, 128)
    assert tvq.tvq_bits_per_element_config(cfg, 1) == pytest.approx((120 + 88) * 8 / 256)
    assert tvq.tvq_bits_per_element_config(cfg, 0) == pytest.approx(6.5)
    # non-power-of-two n is fractional in the paper's accounting, whole bits in storage
    cfg48 = _cfg(tvq, [(48, 48, 32, 32, 0, 0)], 1, 1, 128)
    assert tvq.tvq_bits_per_element_config(cfg48, 0) == pytest.approx(np.log2(48) / 2 + 16)
    assert tvq.tvq_bits_per_element_config(cfg48, 1) == pytest.approx(3.0 + 16)
    assert tvq.tvq_bits_per_element_config(cfg48, 7) < 0


@pytest.mark.parametrize("bad", [
    dict(L=0), dict(L=257), dict(H=0), dict(d=48), dict(d=0), dict(nk=1), dict(nk=4097),
    dict(bk=0, mk=1), dict(bk=17, mk=1), dict(mk=3), dict(signs_bad=True),
])
def test_invalid_configs_rejected_before_gpu(tvq, bad):
    """Config validation is host-only: bad values return TVQ_ERR_INVALID_ARG without a GPU."""
    L = bad.get("L", 2)
    d = bad.get("d", 128)
    nk = bad.get("nk", 64)
    table = [(nk, 64, bad.get("bk", 8), 4, bad.get("mk", 1), 2)] * max(L, 1)
    if L > 256:
        table = table[:256]   # the count is rejected before the table is read
    signs = None
    if bad.get("signs_bad"):
        signs = np.ones((L, d), np.int8)
        signs[1, 3] = 0
    cfg = _cfg(tvq, table, L, bad.get("H", 8), d, signs=signs)
    h = ctypes.c_void_p()
    assert tvq.load_library().tvq_create(ctypes.byref(cfg), ctypes.byref(h)) == -1
    assert not h.value
    lay = tvq.tvq_layout()
    assert tvq.load_library().tvq_layout_for_config(ctypes.byref(cfg), 1, 16, ctypes.byref(lay)) == -1


def test_unsupported_head_dim(tvq):
    """d = 32 and 256 are valid for the method but the GPU kernels are built for 64 and 128."""
    for d in (32, 256):
        cfg = _cfg(tvq, [(64, 64, 8, 4, 1, 2)], 1, 1, d)
        h = ctypes.c_void_p()
        assert tvq.load_library().tvq_create(ctypes.byref(cfg), ctypes.byref(h)) == -2
        assert tvq.tvq_layout_for_config(cfg, 1, 4).total_bytes > 0


def test_null_codec_calls_rejected(tvq):
    lib = tvq.load_library()
    desc = tvq.tvq_tensor_desc(1, 1, 0, 0, 0, 128)
    lay = tvq.tvq_layout()
    assert lib.tvq_encode(None, 0, None, None, ctypes.byref(desc), 0, None, ctypes.byref(lay), None) == -1
    assert lib.tvq_decode(None, None, ctypes.byref(lay), 0, 1, 0, None, None, ctypes.byref(desc), None) == -1
    assert lib.tvq_cache_layout(None, 1, 1, ctypes.byref(lay)) == -1
    assert lib.tvq_bits_per_element(None, 0) < 0
    lib.tvq_destroy(None)


def test_group_packing_storage(tvq):
    """Group packing at n = 48 (d = 128): 45-byte angle records instead of 48, and the
    actual-storage rate drops by 3 * 8 / 128 bits per element; powers of two are unchanged;
    an unknown packing value is rejected."""
    t48 = [(48, 64, 8, 4, 1, 2)]
    plain = tvq.tvq_layout_for_config(_cfg(tvq, t48, 1, 8, 128), 1, 16)
    packed = tvq.tvq_layout_for_config(_cfg(tvq, t48, 1, 8, 128, packing=1), 1, 16)
    assert plain.rec_bytes[0][0][0] == 48 and packed.rec_bytes[0][0][0] == 45
    assert plain.rec_bytes[0][1][0] == packed.rec_bytes[0][1][0] == 48     # n = 64
    r0 = tvq.tvq_bits_per_element_config(_cfg(tvq, t48, 1, 8, 128), 1)
    r1 = tvq.tvq_bits_per_element_config(_cfg(tvq, t48, 1, 8, 128, packing=1), 1)
    assert r0 - r1 == pytest.approx(3 * 8 / 128 / 2)        # averaged over K and V
    assert tvq.tvq_bits_per_element_config(_cfg(tvq, t48, 1, 8, 128, packing=2), 1) < 0


def test_layout_limits(tvq):
    cfg = _cfg(tvq, [(64, 64, 8, 4, 1, 2)], 1, 8, 128)
    lib = tvq.load_library()
    lay = tvq.tvq_layout()
    assert lib.tvq_layout_for_config(ctypes.byref(cfg), 0, 16, ctypes.byref(lay)) == -1
    assert lib.tvq_layout_for_config(ctypes.byref(cfg), 1, 0, ctypes.byref(lay)) == -1
    assert lib.tvq_layout_for_config(ctypes.byref(cfg), 1 << 20, 1 << 12, ctypes.byref(lay)) == -1
    # the largest cache: batch x heads x capacity just below 2^31 slots, sizes in 64 bits
    assert lib.tvq_layout_for_config(ctypes.byref(cfg), (1 << 28) - 1, 1, ctypes.byref(lay)) == 0
    slots = ((1 << 28) - 1) * 8
    assert lay.total_bytes == slots * (120 + 88) and lay.total_bytes > 1 << 38
    assert lay.off[0][1][0] == slots * 120               # V angle plane after K's three
    assert lib.tvq_layout_for_config(ctypes.byref(cfg), 1 << 28, 1, ctypes.byref(lay)) == -1


def _bins_code(code, bound, n, a, b, rcp_ulps=0):
    """The fast encode kernels' table-driven angle code, step by step in fp32 (the reciprocal
    correctly rounded, optionally moved by `rcp_ulps` units in the last place, as the
    hardware's may be); also returns the table index, for bounds checks."""
    a = np.asarray(a, np.float32)
    b = np.asarray(b, np.float32)
    s = (np.abs(a) + np.abs(b)).astype(np.float32)
    r = (np.float32(1.0) / s).astype(np.float32)
    for _ in range(abs(rcp_ulps)):
        r = np.nextafter(r, np.float32(np.inf if rcp_ulps > 0 else 0)).astype(np.float32)
    sa = a.view(np.uint32) >> np.uint32(31)
    r = (r.view(np.uint32) | (sa << np.uint32(31))).view(np.float32)
    p = (b * r).astype(np.float32)
    half = (n - 3) / 2.0
    # fma(p, K/2, K/2 + 1/2 + 1.5 * 2^23): exact in fp64, then rounded once to fp32
    v = (p.astype(np.float64) * half + (half + 0.5 + 12582912.0)).astype(np.float32)
    entry = v.view(np.uint32).astype(np.int64) - 0x4B400000
    idx = entry + (sa.astype(np.int64) << int(np.log2(n)))
    k = (code[idx] + (p >= bound[idx])) % n
    return k.astype(np.int64), entry


@pytest.mark.parametrize("n", [16, 64, 256])
def test_angle_bins_reproduce_the_angle_code(tvq, orc, n):
    """The angle bins of the fast encode kernels (p' = sign(a) b / (|a| + |b|), a cell of
    [-1, 1] per sign of a, the code at the cell's low edge plus one past its boundary) give
    the oracle's code round(n theta / 2 pi) mod n for every pair outside the 1e-6-turn flag
    zone: random directions at scales 2^-40 .. 2^40, the neighbourhoods of every bin boundary,
    the axes (signed zeros included) and the diagonals, with the reciprocal exact or one ulp
    off either way.  The entry index stays inside the half table."""
    code, bound = tvq.tvq_make_angle_bins(n)
    assert code.shape == (2 * n,) and (code < n).all()
    rng = np.random.default_rng(7 + n)
    th = [rng.uniform(-np.pi, np.pi, 200000)]
    edges = (np.arange(n) + 0.5) * 2 * np.pi / n
    for off in (-1e-4, -1e-5, -3e-6, 0.0, 3e-6, 1e-5, 1e-4):
        th.append(edges + off)
    th.append(np.arange(8) * np.pi / 4)
    th = np.concatenate(th)
    scale = 2.0 ** rng.uniform(-40, 40, th.size)
    a = (np.cos(th) * scale).astype(np.float32)
    b = (np.sin(th) * scale).astype(np.float32)
    z = np.float32(0.0)
    axes_a = np.array([1, -1, z, -z, 3e-20, -3e-20, 1, 1, -1, -1], np.float32)
    axes_b = np.array([z, z, 1, -1, z, -z, -z, 1, 1, -1], np.float32)
    a = np.concatenate([a, axes_a])
    b = np.concatenate([b, axes_b])
    u = n * np.arctan2(b.astype(np.float64), a.astype(np.float64)) / (2 * np.pi)
    want = np.mod(np.floor(u + 0.5), n).astype(np.int64)
    for i in rng.choice(u.size, 200, replace=False):
        assert want[i] == orc.angle_code(float(u[i]), n)
    ok = ~orc.angle_flags(u, n)
    for ulps in (0, 1, -1):
        got, entry = _bins_code(code, bound, n, a, b, ulps)
        assert entry.min() >= 0 and entry.max() <= n - 2
        bad = np.nonzero(ok & (got != want))[0]
        assert bad.size == 0, (n, ulps, bad[:5], a[bad[:5]], b[bad[:5]], got[bad[:5]], want[bad[:5]])


def test_angle_bins_reject_other_n(tvq):
    lib = tvq.load_library()
    buf = np.zeros(1024, np.uint32)
    fb = np.zeros(1024, np.float32)
    for n in (8, 48, 512, 0):
        assert lib.tvq_make_angle_bins(n, buf.ctypes.data_as(ctypes.c_void_p),
                                       fb.ctypes.data_as(ctypes.c_void_p)) == -1
    assert lib.tvq_make_angle_bins(64, None, None) == -1


def test_binding_raises_without_the_library(tmp_path):
    """A copy of the package without libtvq.so: constructing a codec raises ImportError naming
    the missing library (there is no fallback path to run instead)."""
    import shutil
    import subprocess
    import sys
    src = os.path.join(ROOT, "paper_2603_27467_amd")
    dst = tmp_path / "paper_2603_27467_amd"
    shutil.copytree(src, dst, ignore=shutil.ignore_patterns("*.so", "*.so.*", "csrc",
                                                            "__pycache__"))
    code = ("import paper_2603_27467_amd as t\n"
            "try:\n"
            "    t.Codec(1, 1, 128, [t.LayerCfg(64, 64)])\n"
            "except ImportError as e:\n"
            "    print('raised:', e)\n"
            "else:\n"
            "    print('no error')\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=tmp_path, capture_output=True,
                       text=True, timeout=120, env={**os.environ, "PYTHONPATH": str(tmp_path)})
    assert r.returncode == 0, r.stderr
    assert r.stdout.startswith("raised:") and "libtvq.so is missing" in r.stdout, r.stdout


def test_binding_checks_extents_before_any_call(tvq):
    """The binding rejects, before it calls the library, tensors whose layers, heads or head
    dim differ from the codec's, caches and pools smaller than their layout, and queries of
    another head dim: the kernels size their accesses from the codec and the layout, so such a
    tensor would be read or written past its end.  (A codec object without a device handle
    stands in for a live one; each call must fail in the binding.)"""
    import torch
    c = tvq.Codec.__new__(tvq.Codec)
    c.L, c.H, c.d, c.handle = 2, 4, 128, 0
    lay = tvq.tvq_layout()
    lay.total_bytes, lay.batch, lay.capacity_tokens = 4096, 1, 8
    cache = torch.zeros(4096, dtype=torch.uint8)
    good = torch.zeros((2, 1, 4, 8, 128), dtype=torch.bfloat16)
    for bad in (torch.zeros((1, 1, 4, 8, 128), dtype=torch.bfloat16),     # fewer layers
                torch.zeros((2, 1, 3, 8, 128), dtype=torch.bfloat16),     # fewer heads
                torch.zeros((2, 1, 4, 8, 64), dtype=torch.bfloat16)):     # other head dim
        with pytest.raises(ValueError, match="codec needs"):
            c.encode(bad, bad, cache, lay)
        with pytest.raises(ValueError, match="codec needs"):
            c.decode(cache, lay, 0, 8, bad, bad)
    for small in (torch.zeros(4095, dtype=torch.uint8), torch.zeros(4096, dtype=torch.int8),
                  torch.zeros(8192, dtype=torch.uint8)[::2]):
        with pytest.raises(ValueError, match="cache"):
            c.encode(good, good, small, lay)
        with pytest.raises(ValueError, match="cache"):
            c.decode(small, lay, 0, 8, good, good)
    q = torch.zeros((1, 8, 64))
    with pytest.raises(ValueError, match="head dim"):
        c.attention(cache, lay, 0, 8, q, torch.zeros_like(q), 0.1)
    q = torch.zeros((1, 8, 128))
    with pytest.raises(ValueError, match="cache"):
        c.attention(torch.zeros(100, dtype=torch.uint8), lay, 0, 8, q, torch.zeros_like(q), 0.1)


def test_header_is_c99_and_host_calls_work_from_c(tvq, tmp_path):
    """include/tvq.h compiles as strict C99, and a C program linked against the library gets
    the layout, rates, signs and refusals its own checks expect (tests/native/abi_c99.c)."""
    import shutil
    import subprocess
    cc = shutil.which("gcc")
    if cc is None:
        pytest.skip("gcc not found")
    lib = tvq.library_path()
    exe = str(tmp_path / "abi_c99")
    subprocess.run([cc, "-std=c99", "-pedantic", "-Wall", "-Wextra", "-Werror",
                    "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "native", "abi_c99.c"), lib,
                    "-Wl,-rpath," + os.path.dirname(lib), "-o", exe], check=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr
