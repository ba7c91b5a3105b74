"""Host-only fuzz of the planners (no GPU): random and extreme extents,
leading dimensions, alignments, kernels and k-slice counts must give a
status, never a crash, and every plan they accept must satisfy the launch
invariants the kernels rely on."""
import numpy as np
import pytest

import paper_2302_07594_amd as ig

BIG = [0, 1, 2, 7, 63, 64, 65, 255, 256, 1000, 4096, 32768, 32769, 70000, (1 << 31) - 1,
       1 << 31, (1 << 40), (1 << 62)]


def _pick(rng, values, p_extreme=0.2):
    if rng.random() < p_extreme:
        return int(rng.choice(values))
    return int(rng.integers(0, 5000))


@pytest.mark.parametrize("seed", range(4))
def test_gemm_plan_invariants(seed):
    rng = np.random.default_rng(seed)
    nk = ig.igemm_num_kernels()
    for _ in range(1500):
        es = int(rng.choice([1, 2]))
        m, n, k = (_pick(rng, BIG) for _ in range(3))
        lda = k + int(rng.integers(0, 3)) * int(rng.choice([0, 1, 8, 1000]))
        ldb = n + int(rng.integers(0, 3)) * int(rng.choice([0, 1, 8, 1000]))
        ldc = n + int(rng.integers(0, 3)) * int(rng.choice([0, 1, 8]))
        base = 0x10000 + int(rng.choice([0, 1, 2, 4, 16]))
        kernel = int(rng.integers(-1, nk))
        split = int(rng.choice([-1, -1, 1, 2, 3, 64, 1 << 20]))
        try:
            p = ig.igemm_query_plan(es, m, n, k, base, max(lda, 1), base, max(ldb, 1), base,
                                    max(ldc, 1), 256, kernel, split)
        except ig.IgemmError as e:
            assert e.status in (ig.IGEMM_EINVAL, ig.IGEMM_ENOTSUP)
            continue
        if m == 0 or n == 0 or k == 0:
            assert p["kernel"] == -1 or p["grid"] >= 0
            continue
        assert 0 <= p["kernel"] < nk
        assert ig.igemm_kernel_name(p["kernel"]).startswith("i16" if es == 2 else "i8")
        assert p["split"] >= 1 and p["k_chunk"] >= 1
        assert p["split"] * p["k_chunk"] >= k
        assert p["k_chunk"] <= 32768
        assert 1 <= p["grid"] < (1 << 32) // 256
        if not p["packed"]:
            assert p["workspace_bytes"] == 0


@pytest.mark.parametrize("seed", range(3))
def test_conv_plan_statuses(seed):
    rng = np.random.default_rng(100 + seed)
    for _ in range(1500):
        vals = [_pick(rng, BIG, 0.15) % 300 if rng.random() < 0.8 else _pick(rng, BIG, 1.0)
                for _ in range(13)]
        n, h, w, c, k, r, s, sh, sw, ph, pw, dh, dw = vals
        # mostly valid small shapes, sometimes extreme or invalid ones
        if rng.random() < 0.7:
            r, s = 1 + r % 7, 1 + s % 7
            sh, sw, dh, dw = 1 + sh % 3, 1 + sw % 3, 1 + dh % 3, 1 + dw % 3
            ph, pw = ph % 4, pw % 4
        d = ig.conv_desc(n, h, w, c, k, r, s, (sh, sw), (ph, pw), (dh, dw))
        es = int(rng.choice([1, 2]))
        try:
            p = ig.igemm_conv2d_query_plan(es, d)
        except ig.IgemmError as e:
            assert e.status in (ig.IGEMM_EINVAL, ig.IGEMM_ENOTSUP)
            continue
        if p["kernel"] < 0:
            continue
        oh = ig.igemm_conv2d_out_dim(h, r, sh, ph, dh)
        ow = ig.igemm_conv2d_out_dim(w, s, sw, pw, dw)
        assert oh > 0 and ow > 0 and n > 0 and k > 0 and c > 0
        kk = r * s * c
        assert p["split"] * p["k_chunk"] >= kk and p["k_chunk"] <= 32768
        assert 1 <= p["grid"] < (1 << 32) // 256
        assert not p["packed"]


@pytest.mark.parametrize("fn", [ig.igemm_i16_srs, ig.igemm_i8_srs])
def test_srs_status_only_without_device(fn):
    """Arguments that fail validation or planning return before any HIP call,
    so these run on a machine without a GPU."""
    rng = np.random.default_rng(7)
    for _ in range(1000):
        m, n = _pick(rng, BIG, 0.3), _pick(rng, BIG, 0.3)
        k = int(rng.choice([40000, 1 << 31, 1 << 40, 70000]))
        kc = int(rng.choice([-5, 0, 32769, 1 << 20]))
        shift = int(rng.choice([-1, 48, 100]))
        st = fn(max(m, 1), max(n, 1), k, 0x10000, k, 0x20000, max(n, 1), 0x30000, max(n, 1),
                kc, shift, 0, 0)
        assert st in (ig.IGEMM_EINVAL, ig.IGEMM_ENOTSUP)


@pytest.mark.parametrize("seed", range(2))
def test_srs_query_invariants(seed):
    """The int16-output workspace query: a status for any arguments; when it
    accepts them, the bytes are those of the packed plan of the same product
    plus two words per padded row and column and block, or 0 (fused path),
    and never more than 0 for int8 operands or for blocks the packed path
    cannot take."""
    rng = np.random.default_rng(100 + seed)
    nk = ig.igemm_num_kernels()
    for _ in range(1500):
        es = int(rng.choice([1, 2]))
        m, n, k = (_pick(rng, BIG) for _ in range(3))
        kc = int(rng.choice([0, 0, 1, 100, 256, 512, 290, 32768, 32769, -1, k + 3]))
        kernel = int(rng.integers(-1, nk))
        num_cu = int(rng.choice([0, 1, 80, 256, 304]))
        try:
            need = ig.igemm_srs_query(es, m, n, k, 0x10000, max(k, 1), 0x10000, max(n, 1),
                                      0x10000, max(n, 1), kc, num_cu, kernel)
        except ig.IgemmError as e:
            assert e.status in (ig.IGEMM_EINVAL, ig.IGEMM_ENOTSUP)
            continue
        assert need >= 0
        if need == 0:
            continue
        blk = k if kc == 0 or kc > k else kc
        nblocks = -(-k // blk)
        assert es == 2 and nblocks <= 64 and (nblocks == 1 or blk % 256 == 0)
        p = ig.igemm_query_plan(es, m, n, k, 0x10000, max(k, 1), 0x10000, max(n, 1), 0x10000,
                                max(n, 1), num_cu, kernel if kernel >= 0 else -1)
        assert p["packed"]
        m_pad, n_pad = -(-m // 128) * 128, -(-n // 128) * 128
        assert need == p["workspace_bytes"] + 8 * nblocks * (m_pad + n_pad)
