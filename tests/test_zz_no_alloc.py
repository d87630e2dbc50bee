"""viscache_decode_step_noalloc, the decode step for callers that cannot
allocate device memory, against viscache_decode_step (same kernels, so bit for
bit) through the C ABI: two calls in a row, the second with a smaller input,
and several steps on one cache; sizes beyond its scratch are refused on the
host."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_24063_amd as vc
    vc.lib()
    return torch.device("cuda:0")


def _pair(dev, sg, seed, L, B, Hq, Hkv, d, lens, extra):
    """Two caches with the same contents and lengths."""
    from paper_2608_24063_amd.tensors import DecodeCache
    from synthgen.device import bf16_tensor
    caps = [x + extra for x in lens]
    cs = []
    for _ in range(2):
        c = DecodeCache(L, B, Hq, Hkv, d, caps, dev)
        c.k_pool.copy_(bf16_tensor(sg.normal_bf16(seed, 1, (c.total_rows, d)), dev))
        c.v_pool.copy_(bf16_tensor(sg.normal_bf16(seed, 2, (c.total_rows, d)), dev))
        c.len.copy_(torch.tensor(lens, dtype=torch.int32))
        cs.append(c)
    return cs


def _steps(dev, sg, seed, L, B, Hq, Hkv, d, lens, steps):
    from synthgen.device import bf16_tensor
    a, b = _pair(dev, sg, seed, L, B, Hq, Hkv, d, lens, steps)
    kn = bf16_tensor(sg.normal_bf16(seed, 3, (steps, L, B, Hkv, d)), dev)
    vn = bf16_tensor(sg.normal_bf16(seed, 4, (steps, L, B, Hkv, d)), dev)
    q = bf16_tensor(sg.normal_bf16(seed, 5, (steps, L, B, Hq, d)), dev)
    oa = torch.full((L, B, Hq, d), float("nan"), dtype=torch.float32, device=dev)
    ob = torch.full((L, B, Hq, d), float("nan"), dtype=torch.float32, device=dev)
    for t in range(steps):
        a.step(kn[t], vn[t], q[t], oa, d ** -0.5)
        b.step_noalloc(kn[t], vn[t], q[t], ob, d ** -0.5)
        torch.cuda.synchronize()
        assert torch.equal(oa, ob), f"step {t}: outputs differ"
    assert torch.equal(a.len, b.len)
    assert torch.equal(a.k_pool.view(torch.int16), b.k_pool.view(torch.int16))
    assert torch.equal(a.v_pool.view(torch.int16), b.v_pool.view(torch.int16))
    assert not torch.isnan(ob).any()


def test_noalloc_matches_step_then_smaller(dev, sg):
    # First call: 48 units with long, split caches (many pieces, merges);
    # second: a smaller shape whose counters and partials reuse the front of
    # the same scratch.
    lens = [0, 1, 31, 33, 3100, 511, 1023, 1024, 1100, 5, 64, 2049, 2, 1025, 47, 4097] * 3
    _steps(dev, sg, 21, 3, 2, 32, 8, 128, lens, 2)
    _steps(dev, sg, 22, 2, 1, 8, 2, 64, [7, 300, 0, 65], 2)


def test_noalloc_many_steps_pruned_shape(dev, sg):
    # 7B-like decode shape: 28 layers x 4 kv heads, kept rows of a pruned
    # cache plus a 64-row window, several steps with appends.
    rng = np.random.default_rng(5)
    lens = [int(x) for x in rng.integers(700, 1480, 28 * 4)]
    _steps(dev, sg, 23, 28, 1, 28, 4, 128, lens, 6)


def test_noalloc_refuses_beyond_its_scratch(dev):
    import paper_2608_24063_amd as vc
    from paper_2608_24063_amd.tensors import DecodeCache
    # one unit more than the scratch has counters for
    units = vc.VC_DECODE_NOALLOC_UNITS + 1
    c = DecodeCache(1, units, 1, 1, 64, [1] * units, dev)
    kn = torch.zeros((units, 64), dtype=torch.bfloat16, device=dev)
    q = torch.zeros((units, 64), dtype=torch.bfloat16, device=dev)
    out = torch.zeros((units, 64), dtype=torch.float32, device=dev)
    with pytest.raises(vc.VisCacheError) as ei:
        c.step_noalloc(kn, kn, q, out, 0.125)
    assert ei.value.status == vc.VC_ERR_WORKSPACE
