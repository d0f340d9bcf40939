"""Host-side checks of the C ABI (no GPU needed): the library loads, exports every
function include/dash.h declares, and rejects bad arguments before any HIP call.
Also checks the HIP path's float32 sampler arithmetic, built for the host, bit for
bit against the oracle."""
import ctypes as C
import os
import re
import shutil
import subprocess

import numpy as np
import pytest

from oracle import sampler as osm
from paper_2505_17218_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dash.h")

pytestmark = pytest.mark.skipif(not os.path.exists(L.LIB_PATH), reason="libdash.so not built")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dash_[a-z0-9_]+)\s*\(", src)))


def test_header_symbols_exported():
    lib = L.load()
    names = declared_functions()
    assert len(names) >= 20
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(L.header_functions())


def test_version_and_status_strings():
    assert L.dash_abi_version() == 2
    lib = L.load()
    for s in range(6):
        assert lib.dash_status_str(s)
    assert lib.dash_status_str(99) == b"unknown status"


def _desc(**kw):
    base = dict(n_layers=2, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16, d_ff=172, vocab=512, dtype=0,
                rope_theta=1e4, rms_eps=1e-6)
    base.update(kw)
    return L.dash_model_desc(*[base[k] for k, _ in L.dash_model_desc._fields_])


def _fake_ptrs(desc):
    n = L.dash_weight_count(desc)
    return [0x10000 * (i + 1) if i != 2 else None for i in range(n)]


def test_model_create_validation():
    d = _desc()
    h = L.dash_model_create(d, _fake_ptrs(d))  # no device access at creation
    assert h
    assert L.dash_workspace_bytes(h, 16, 48) > 0
    L.dash_model_destroy(h)
    cases = [(_desc(n_heads=3), L.DASH_EINVAL), (_desc(head_dim=15), L.DASH_EINVAL),
             (_desc(dtype=1, head_dim=16), L.DASH_ENOTSUP), (_desc(dtype=7), L.DASH_EINVAL),
             (_desc(n_layers=0), L.DASH_EINVAL), (_desc(head_dim=256), L.DASH_ENOTSUP)]
    for d2, want in cases:
        n = L.dash_weight_count(d2)
        ptrs = [0x10000 * (i + 1) if i != 2 else None for i in range(max(n, 1))]
        with pytest.raises(L.DashError) as e:
            L.dash_model_create(d2, ptrs)
        assert e.value.status == want, (d2.n_heads, d2.head_dim, d2.dtype)
    with pytest.raises(L.DashError) as e:
        L.dash_model_create(d, _fake_ptrs(d)[:-1])
    assert e.value.status == L.DASH_EINVAL
    p = _fake_ptrs(d)
    p[5] = 0x10004  # misaligned
    with pytest.raises(L.DashError) as e:
        L.dash_model_create(d, p)
    assert e.value.status == L.DASH_EINVAL
    p = _fake_ptrs(d)
    p[2] = 0x20000  # untied lm head
    with pytest.raises(L.DashError) as e:
        L.dash_model_create(d, p)
    assert e.value.status == L.DASH_ENOTSUP


def test_sample_and_advantage_validation():
    with pytest.raises(L.DashError) as e:
        L.dash_sample(0x1000, 512, 4, 512, None, 0x2000, 0x3000, 0.0, 1, 0x4000, None, None, None, None)
    assert e.value.status == L.DASH_EINVAL
    with pytest.raises(L.DashError) as e:
        L.dash_sample(0x1000, 100, 4, 512, None, 0x2000, 0x3000, 1.0, 1, 0x4000, None, None, None, None)
    assert e.value.status == L.DASH_EINVAL
    with pytest.raises(L.DashError) as e:
        L.dash_sample(0x1000, 512, 4, 512, None, 0x2000, 0x3000, float("nan"), 1, 0x4000, None, None, None, None)
    assert e.value.status == L.DASH_EINVAL
    # zero rows is a no-op, not an error
    L.dash_sample(0x1000, 512, 0, 512, None, 0x2000, 0x3000, 1.0, 1, 0x4000, None, None, None, None)
    for args, want in [((0, 4), L.DASH_EINVAL), ((4, 0), L.DASH_EINVAL), ((1, 65537), L.DASH_ENOTSUP),
                       ((1 << 20, 64), L.DASH_ENOTSUP)]:
        with pytest.raises(L.DashError) as e:
            L.dash_group_advantage_filter(0x1000, args[0], args[1], 2, 1e-6, 0.1, 0x2000, 0x3000, 0x4000, None)
        assert e.value.status == want
    for mode, eps, tau in [(4, 1e-6, 0.1), (-1, 1e-6, 0.1), (2, -1.0, 0.1), (2, 1e-6, float("nan"))]:
        with pytest.raises(L.DashError) as e:
            L.dash_group_advantage_filter(0x1000, 4, 4, mode, eps, tau, 0x2000, 0x3000, 0x4000, None)
        assert e.value.status == L.DASH_EINVAL
    with pytest.raises(L.DashError) as e:  # leave-one-out needs a second sample
        L.dash_group_advantage_filter(0x1000, 4, 1, L.DASH_ADV_LOO, 0.0, 0.1, 0x2000, 0x3000, 0x4000, None)
    assert e.value.status == L.DASH_EINVAL


def test_recompute_loss_and_profiler_validation():
    d = _desc()
    h = L.dash_model_create(d, _fake_ptrs(d))
    # workspace of the teacher-forced recompute grows with the chunk; 0 for bad sizes
    w1 = L.dash_teacher_forced_workspace_bytes(h, 1, 48, 16)
    w4 = L.dash_teacher_forced_workspace_bytes(h, 4, 48, 16)
    assert 0 < w1 < w4
    assert w4 >= 4 * 32 * d.vocab * 4  # the chunk's logits: 4 sequences x 32 scored positions
    assert L.dash_teacher_forced_workspace_bytes(h, 1, 16, 16) == 0  # nothing to score
    assert L.dash_teacher_forced_workspace_bytes(h, 0, 48, 16) == 0
    with pytest.raises(L.DashError) as e:  # no kv handle
        L.dash_teacher_forced_logprobs(h, None, 0x1000, 2, 48, 16, 0x2000, 0x3000, w1, None)
    assert e.value.status == L.DASH_EINVAL
    L.dash_model_destroy(h)
    for args in [(None, 8, 8, None, 0x2000, 0x3000, 0x4000, 4, 0x5000, None),   # no log-probs
                 (0x1000, 4, 8, None, 0x2000, 0x3000, 0x4000, 4, 0x5000, None),  # ld < T
                 (0x1000, 8, 0, None, 0x2000, 0x3000, 0x4000, 4, 0x5000, None),  # T = 0
                 (0x1000, 8, 8, None, 0x2000, 0x3000, 0x4000, 0, 0x5000, None)]:  # n_total = 0
        with pytest.raises(L.DashError) as e:
            L.dash_pg_loss(*args, None)
        assert e.value.status == L.DASH_EINVAL
    with pytest.raises(L.DashError) as e:
        L.dash_profile_layer(-2)
    assert e.value.status == L.DASH_EINVAL
    L.dash_profile_layer(-1)
    with pytest.raises(L.DashError) as e:
        L.dash_kv_split_keys(None)
    assert e.value.status == L.DASH_EINVAL


def test_kl_and_policy_loss_validation():
    d = _desc()
    h = L.dash_model_create(d, _fake_ptrs(d))
    # the teacher-forced KL keeps two logits buffers per chunk
    w1 = L.dash_teacher_forced_kl_workspace_bytes(h, 1, 48, 16)
    assert w1 >= L.dash_teacher_forced_workspace_bytes(h, 1, 48, 16) + 32 * d.vocab * 4
    assert L.dash_teacher_forced_kl_workspace_bytes(h, 1, 16, 16) == 0
    assert L.dash_teacher_forced_kl_workspace_bytes(h, 0, 48, 16) == 0
    for base, kv in [(None, 0x100), (h, None)]:
        with pytest.raises(L.DashError) as e:  # NULL base / kv handle
            L.dash_teacher_forced_kl(h, base, kv, 0x1000, 2, 48, 16, None, 0x2000, None, 0x3000, w1, None)
        assert e.value.status == L.DASH_EINVAL
    L.dash_model_destroy(h)
    for args in [(None, 0x2000, 8, 4, 8),    # no theta logits
                 (0x1000, 0x2000, 4, 4, 8),  # ld < vocab
                 (0x1000, 0x2000, 8, 4, 0),  # empty vocabulary
                 (0x1000, 0x2000, 8, -1, 8)]:  # negative row count
        with pytest.raises(L.DashError) as e:
            L.dash_logits_kl(args[0], args[1], args[2], args[3], args[4], 0x3000, None, None)
        assert e.value.status == L.DASH_EINVAL
    base = (0x1000, 0x1100, 0x1200, 8, 8, None, 0x2000, 0x3000, 0x4000, 4)
    for change, eps, beta in [({0: None}, 0.2, 0.0), ({3: 4}, 0.2, 0.0), ({9: 0}, 0.2, 0.0),
                              ({}, 1.0, 0.0), ({}, -0.1, 0.0), ({}, float("nan"), 0.0), ({}, 0.2, float("inf"))]:
        a = list(base)
        for i, v in change.items():
            a[i] = v
        with pytest.raises(L.DashError) as e:
            L.dash_policy_loss(*a, eps, beta, 0x5000, None, None)
        assert e.value.status == L.DASH_EINVAL


def test_kv_sizes():
    d = _desc()
    h = L.dash_model_create(d, _fake_ptrs(d))
    # page = layers * kv heads * (K, V) * page_size * head_dim * 4 bytes
    assert L.dash_kv_page_bytes(h, 16) == 2 * 2 * 2 * 16 * 16 * 4
    assert L.dash_kv_table_bytes(16, 48, 16) >= 16 * 3 * 4 + 4
    L.dash_model_destroy(h)


@pytest.fixture(scope="module")
def host_math(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    exe = str(tmp_path_factory.mktemp("hm") / "hm")
    src = os.path.join(ROOT, "tests", "hip_sampler_math_host.cpp")
    inc = os.path.join(ROOT, "paper_2505_17218_amd", "csrc")
    subprocess.run([hipcc, "-O2", "-ffp-contract=off", "-I", inc, src, "-o", exe], check=True,
                   capture_output=True, timeout=300)

    def run(lines):
        out = subprocess.run([exe], input="\n".join(lines) + "\n", capture_output=True, text=True, check=True)
        return out.stdout.split("\n")
    return run


def test_hip_sampler_math_matches_oracle_bitwise(host_math):
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.random(3000, dtype=np.float32) * np.float32(2) + np.float32(1e-3),
                        np.exp(rng.uniform(-80, 80, 3000)).astype(np.float32),
                        np.arange(1, 200, dtype=np.float32) * np.float32(2.0 ** -24),
                        np.array([1.0, 2.0, 0.5, 1.4142135, 1.4142137, 0.70710677], np.float32)])
    out = host_math([f"log {b:08x}" for b in x.view(np.uint32)])
    got = np.array([int(o, 16) for o in out if o], dtype=np.uint32)
    np.testing.assert_array_equal(got, osm.own_log(x).view(np.uint32))
    bits = rng.integers(0, 2 ** 32, 5000, dtype=np.uint64).astype(np.uint32)
    bits[:4] = [0, 0xFFFFFFFF, 0x80000000, 0xFF]
    out = host_math([f"gumbel {b:08x}" for b in bits])
    got = np.array([int(o, 16) for o in out if o], dtype=np.uint32)
    np.testing.assert_array_equal(got, osm.gumbel_from_bits(bits).view(np.uint32))
    ctr = rng.integers(0, 2 ** 32, (200, 4), dtype=np.uint64).astype(np.uint32)
    key = rng.integers(0, 2 ** 32, (200, 2), dtype=np.uint64).astype(np.uint32)
    out = host_math([" ".join(f"{v:08x}" for v in (*c, *k)) .join(["philox ", ""]) for c, k in zip(ctr, key)])
    got = np.array([[int(w, 16) for w in o.split()] for o in out if o], dtype=np.uint32)
    want = np.stack([osm.philox4x32_10(c[None], (int(k[0]), int(k[1])))[0] for c, k in zip(ctr, key)])
    np.testing.assert_array_equal(got, want)
