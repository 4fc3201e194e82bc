"""CPU checks of the seeded input draws: the counter-based stream used for
device-drawn expert pools is Philox4x64-10 as published, element ranges are
independent of how they are chunked, and the values are ~N(0, std)."""
import numpy as np

from paper_2609_34117_amd import inputs as I

MASK = (1 << 64) - 1
# Philox4x64 constants of the published definition (Salmon et al., SC 2011):
# round multipliers and the Weyl key increments
M0, M1 = 0xD2E7470EE14C6C93, 0xCA5A826395121157
W0, W1 = 0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B


def philox4x64_10(ctr, key):
    """Ten rounds: (c0, c1, c2, c3) -> (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2),
    hi(M0 c0) ^ c3 ^ k1, lo(M0 c0)), the key bumped by the Weyl constants
    before every round but the first.  Plain Python integers."""
    c, k = list(ctr), list(key)
    for r in range(10):
        if r:
            k = [(k[0] + W0) & MASK, (k[1] + W1) & MASK]
        p0, p1 = M0 * c[0], M1 * c[2]
        c = [(p1 >> 64) ^ c[1] ^ k[0], p1 & MASK, (p0 >> 64) ^ c[3] ^ k[1], p0 & MASK]
    return c


def element_by_hand(key, i, std):
    b = philox4x64_10([i + 1, 0, 0, 0], [int(key[0]), int(key[1])])
    s = sum((w >> (16 * h)) & 0xFFFF for w in b[:3] for h in range(4))
    v = np.float32(s - 393210) * np.float32(np.float32(std) / np.float32(65536))
    return int(I.to_bf16_bits(np.array([v], np.float32))[0])


def test_numpy_philox_stream_is_the_published_philox4x64_10():
    for key in ([0, 0], [1, 2], [0x0123456789ABCDEF, 0xFEDCBA9876543210], [2 ** 64 - 1, 7]):
        for start in (0, 1, 41, 2 ** 40 + 3):
            bg = np.random.Philox(key=np.array(key, np.uint64),
                                  counter=np.array([start, 0, 0, 0], np.uint64))
            raw = [int(v) for v in bg.random_raw(8)]
            # numpy advances the counter before each block
            want = philox4x64_10([start + 1, 0, 0, 0], key) + philox4x64_10([start + 2, 0, 0, 0], key)
            assert raw == want, (key, start)


def test_elements_follow_the_documented_composition():
    key = I.philox_key(4, 19, I.W13)
    for start, n in ((0, 5), (123456, 3), (2 ** 33 + 5, 2)):
        got = I.philox_normal_bf16(key, start, n, 0.02)
        assert [int(v) for v in got] == [element_by_hand(key, start + j, 0.02) for j in range(n)]
    got = I.philox_normal_bf16(key, 77, 1, 1.0)
    assert int(got[0]) == element_by_hand(key, 77, 1.0)


def test_ranges_do_not_depend_on_chunking():
    key = I.philox_key(4, 0, I.W2)
    whole = I.philox_normal_bf16(key, 1000, 50_000, 0.02)
    parts = np.concatenate([I.philox_normal_bf16(key, 1000, 123, 0.02),
                            I.philox_normal_bf16(key, 1123, 50_000 - 123, 0.02)])
    np.testing.assert_array_equal(whole, parts)
    # different tensors and layers draw different streams
    other = I.philox_normal_bf16(I.philox_key(4, 1, I.W2), 1000, 50_000, 0.02)
    assert not np.array_equal(whole, other)


def test_moments_are_those_of_a_normal():
    v = I.bf16_bits_to_f32(I.philox_normal_bf16(I.philox_key(4, 3, I.W13), 0, 400_000, 0.02))
    assert abs(v.mean()) < 4 * 0.02 / np.sqrt(v.size)
    assert abs(v.std() - 0.02) < 2e-4
    assert np.abs(v).max() <= 6 * 0.02 * 1.01
    # kurtosis of Irwin-Hall(12) is 3 - 1.2/12 = 2.9
    z = (v - v.mean()) / v.std()
    assert abs((z ** 4).mean() - 2.9) < 0.05


def test_expert_slices_are_the_tensor_rows():
    cfg = I.MoEConfig("gen_small", 4, hidden=64, n_experts=6, top_k=2, inter=32, tokens=4)
    w13 = I.philox_expert_slice(cfg, 2, "w13", [1, 4])
    key = I.philox_key(4, 2, I.W13)
    per = 2 * 32 * 64
    np.testing.assert_array_equal(w13[1].ravel(), I.philox_normal_bf16(key, 4 * per, per, 0.02))
    w2 = I.philox_expert_slice(cfg, 2, "w2", [5])
    assert w2.shape == (1, 64, 32)
