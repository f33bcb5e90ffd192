"""GPU parity: every entry point of libw4a8, called through the C ABI, against
the CPU oracle on the same seeded inputs.

Bit-exact: Q8_0 and Q4_0 bytes, int32 block dots (through unit scales), the
routing permutation and counts, and run-to-run determinism.  Floats: within
1e-5 of sum |d_w d_a s| elementwise.  MoE layers: see tests/moe_check.py."""
import numpy as np
import pytest

import oracle
from paper_2606_24031_amd import synth
import paper_2606_24031_amd as w4
from tests import moe_check

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

DEV = "cuda"


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


# ------------------------------------------------------------------ quantizers
def _activation_rows(g, rows, K):
    x = synth.normal_f32(g, (rows, K))
    x *= (2.0 ** g.integers(-8, 8, size=(rows, 1))).astype(np.float32)
    x[g.random((rows, K)) < 0.01] = 0.0
    return x


def _special_rows(K):
    rows = []
    z = np.zeros(K, np.float32); rows.append(z)                              # zero blocks
    t = np.zeros(K, np.float32); t[::32] = 127.0; t[1::32] = 0.5; t[2::32] = -2.5; t[3::32] = 63.5
    rows.append(t)                                                          # exact .5 ties at d = 1
    s = np.full(K, 1.0e-6, np.float32); s[::7] = -3.0e-6; rows.append(s)    # fp16-subnormal scale
    u = np.full(K, 1e-40, np.float32); rows.append(u)                       # fp32 subnormal input
    b = np.full(K, 8.0e6, np.float32); b[::3] = -1.0; rows.append(b)        # large scale
    return np.stack(rows)


@pytest.mark.parametrize("rows,K", [(1, 32), (3, 96), (7, 2048), (129, 512), (1000, 1024)])
def test_q8_0_bit_exact(rows, K):
    g = synth.rng(100 + rows)
    x = np.concatenate([_activation_rows(g, rows, K), _special_rows(K)])
    gpu = host(w4.q8_0_quantize(dev(x)))
    assert np.array_equal(gpu, oracle.q8_0_quantize(x))


@pytest.mark.parametrize("rows,K", [(1, 32), (5, 160), (64, 2048), (1023, 512)])
def test_q4_0_bit_exact(rows, K):
    g = synth.rng(200 + rows)
    w = synth.normal_f32(g, (rows, K), 0.02)
    specials = _special_rows(K)
    specials[2] *= np.float32(0.05)   # |m|/8 below the fp16 normal range: low clamp
    w = np.concatenate([w, specials, -specials])
    gpu = host(w4.q4_0_quantize(dev(w)))
    assert np.array_equal(gpu, oracle.q4_0_quantize(w))


# ------------------------------------------------------------------ gemv
@pytest.mark.parametrize("N,K", [(1024, 1024), (1, 256), (7, 768), (333, 2048),
                                 (64, 16384), (5, 32768), (4097, 512)])
def test_gemv_matches_oracle(N, K):
    g = synth.rng(300 + N)
    W = synth.normal_f32(g, (N, K), 0.02)
    x = synth.normal_f32(g, (K,))
    wq = w4.q4_0_quantize(dev(W))
    xq = w4.q8_0_quantize(dev(x))
    wq_ref, xq_ref = oracle.q4_0_quantize(W), oracle.q8_0_quantize(x)
    assert np.array_equal(host(wq), wq_ref) and np.array_equal(host(xq), xq_ref)
    y = host(w4.q4q8_gemv(wq, xq, N, K))
    y_ref, R = oracle.gemv(wq_ref, xq_ref, N, K)
    assert np.all(np.abs(y - y_ref) <= 1e-5 * R)


@pytest.mark.parametrize("N,K", [(256, 2048), (33, 1024)])
def test_gemv_unit_scales_give_exact_integer_dots(N, K):
    """With every scale 1.0 each partial sum is an integer below 2^24, so the
    fp32 result equals the int32 block-dot sum exactly, in any order."""
    g = synth.rng(400 + N)
    w = synth.q4_0_random_blocks(g, N, K).reshape(N, K // 32, 18)
    w[:, :, 0:2] = np.array([0x3C00], np.uint16).view(np.uint8)
    xq = oracle.q8_0_quantize(synth.normal_f32(g, (K,))).reshape(K // 32, 34)
    xq[:, 0:2] = np.array([0x3C00], np.uint16).view(np.uint8)
    y = host(w4.q4q8_gemv(dev(w), dev(xq), N, K))
    y_ref, _ = oracle.gemv(w, xq, N, K)
    assert np.array_equal(y.astype(np.float64), y_ref)


def test_gemv_lm_head_shape_sampled_rows():
    """The output projection's shape (N = 151936 vocabulary rows, K = 2048):
    random Q4_0 blocks made on the host, 200 sampled rows and the first and
    last rows against the oracle."""
    N, K = 151936, 2048
    g = synth.rng(500)
    w = synth.q4_0_random_blocks(g, N, K).reshape(N, K // 32 * 18)
    x = synth.normal_f32(g, (K,))
    xq = oracle.q8_0_quantize(x)
    y = host(w4.q4q8_gemv(dev(w), dev(xq), N, K))
    rows = np.unique(np.concatenate([[0, N - 1], g.choice(N, 200, replace=False)]))
    y_ref, R = oracle.gemv(w[rows], xq, len(rows), K)
    assert np.all(np.abs(y[rows] - y_ref) <= 1e-5 * R)


def test_gemv_zero_codes_give_zero():
    N, K = 100, 512
    w = np.zeros((N, K // 32, 18), np.uint8)
    w[:, :, 0:2] = np.array([0x2E66], np.uint16).view(np.uint8)
    w[:, :, 2:] = 0x88
    g = synth.rng(5)
    xq = w4.q8_0_quantize(dev(synth.normal_f32(g, (K,))))
    assert not host(w4.q4q8_gemv(dev(w), xq, N, K)).any()


# ------------------------------------------------------------------ MoE layer
class Layer:
    def __init__(self, seed, H, I, E, shared=True):
        g = synth.rng(seed)
        self.H, self.I, self.E = H, I, E
        self.w_gu = synth.q4_0_random_blocks(g, E * 2 * I, H)
        self.w_d = synth.q4_0_random_blocks(g, E * H, I)
        self.ws_gu = synth.q4_0_random_blocks(g, 2 * I, H) if shared else None
        self.ws_d = synth.q4_0_random_blocks(g, H, I) if shared else None
        self.d_gu, self.d_d = dev(self.w_gu), dev(self.w_d)
        self.d_sgu = dev(self.ws_gu) if shared else None
        self.d_sd = dev(self.ws_d) if shared else None
        self.g = g

    def run(self, x, ids, wts, k, ws=None):
        T = x.shape[0]
        if ws is None:
            ws = w4.moe_workspace(T, self.H, self.I, self.E, k)
        out = w4.moe_forward(dev(x), dev(ids), dev(wts), self.d_gu, self.d_d, self.d_sgu,
                             self.d_sd, self.H, self.I, self.E, k, ws)
        lay = w4.moe_workspace_layout(T, self.H, self.I, self.E, k)
        P = T * k + T
        wsn = host(ws)
        h = wsn[lay["h"]:lay["h"] + P * self.I * 4].view(np.float32).reshape(P, self.I)
        hq = wsn[lay["hq"]:lay["hq"] + P * (self.I // 32) * 34].reshape(P, -1)
        perm = wsn[lay["perm"]:lay["perm"] + P * 4].view(np.int32)
        count = wsn[lay["count"]:lay["count"] + self.E * 4].view(np.int32)
        assert not wsn[lay["sync"]:lay["sync_end"]].any(), "sync words not back to zero"
        xq = wsn[lay["xq"]:lay["xq"] + T * (self.H // 32) * 34].reshape(T, -1)
        assert np.array_equal(xq, oracle.q8_0_quantize(x)), "workspace Q8_0(x)"
        return host(out), h, hq, perm, count, ws

    def check(self, x, ids, wts, k, out, h, hq, shared_w=None):
        """The MoE check; at one token no Q8_0(h) block may differ from the
        oracle's own choice (flips are counted and reported otherwise)."""
        return moe_check.check_layer(out, h, hq, x, ids, wts, self.w_gu, self.w_d, self.ws_gu,
                                     self.ws_d, self.H, self.I, self.E, k, shared_w=shared_w,
                                     max_flips=0 if x.shape[0] == 1 else None)


def _check_route(ids, E, shared, perm, count):
    T, k = ids.shape
    flat = ids.ravel()
    valid = (flat >= 0) & (flat < E)
    assert np.array_equal(count, np.bincount(flat[valid], minlength=E)[:E])
    order = np.argsort(np.where(valid, flat, E), kind="stable")[: valid.sum()]
    nr = valid.sum()
    assert np.array_equal(perm[:nr], order)
    if shared:
        assert np.array_equal(perm[nr:nr + T], T * k + np.arange(T))


@pytest.fixture(scope="module")
def small_layer():
    return Layer(7, 256, 256, 4)


def test_moe_small_with_special_routing(small_layer):
    L = small_layer
    g = synth.rng(8)
    T, k = 6, 3
    x = synth.normal_f32(g, (T, L.H))
    ids, wts = synth.routing(g, T, L.E, k)
    ids[1, 2] = -1                 # skipped slot
    ids[2, 1] = ids[2, 0]          # duplicate expert in one token
    ids[3, :] = 2                  # all slots on one expert
    ids[4, 0] = 99                 # id >= E: skipped
    wts[5, :] = 0.0                # shared expert only
    out, h, hq, perm, count, _ = L.run(x, ids, wts, k)
    _check_route(ids, L.E, True, perm, count)
    ids_o = ids.copy(); ids_o[ids_o >= L.E] = -1
    L.check(x, ids_o, wts, k, out, h, hq)


def test_moe_no_shared_expert():
    L = Layer(9, 512, 256, 3, shared=False)
    g = synth.rng(10)
    T, k = 9, 2
    x = synth.normal_f32(g, (T, L.H))
    ids, wts = synth.routing(g, T, L.E, k)
    out, h, hq, perm, count, _ = L.run(x, ids, wts, k)
    _check_route(ids, L.E, False, perm, count)
    L.check(x, ids, wts, k, out, h, hq)


def test_moe_token_without_pairs_gets_zeros():
    """No shared expert and a token whose every slot is skipped (-1, or an id
    >= E): its output row is exactly zero, also where the combine runs in
    the small-group down kernel (T <= 32) and the output buffer held NaN;
    every other row as the oracle."""
    L = Layer(13, 512, 256, 3, shared=False)
    g = synth.rng(14)
    for T in (9, 40):
        k = 2
        x = synth.normal_f32(g, (T, L.H))
        ids, wts = synth.routing(g, T, L.E, k)
        ids[4, :] = -1
        ids[6, 0] = -1
        ids[6, 1] = 77
        ws = w4.moe_workspace(T, L.H, L.I, L.E, k)
        out = torch.full((T, L.H), float("nan"), device="cuda")
        w4.moe_forward(dev(x), dev(ids), dev(wts), L.d_gu, L.d_d, None, None, L.H, L.I, L.E, k,
                       ws, out=out)
        o = host(out)
        assert np.all(o[4] == 0.0) and np.all(o[6] == 0.0)
        lay = w4.moe_workspace_layout(T, L.H, L.I, L.E, k)
        P = T * k + T
        wsn = host(ws)
        h = wsn[lay["h"]:lay["h"] + P * L.I * 4].view(np.float32).reshape(P, L.I)
        hq = wsn[lay["hq"]:lay["hq"] + P * (L.I // 32) * 34].reshape(P, -1)
        ids_o = ids.copy(); ids_o[ids_o >= L.E] = -1
        L.check(x, ids_o, wts, k, o, h, hq)


def test_moe_ragged_group_count_and_odd_K():
    """H = I = 768 (three 8-block groups per row, not a power of two)."""
    L = Layer(11, 768, 768, 5)
    g = synth.rng(12)
    T, k = 7, 2
    x = synth.normal_f32(g, (T, L.H))
    ids, wts = synth.routing(g, T, L.E, k)
    out, h, hq, perm, count, _ = L.run(x, ids, wts, k)
    L.check(x, ids, wts, k, out, h, hq)


@pytest.fixture(scope="module")
def qwen_layer():
    """H=2048, I=512, 256 routed experts + 1 shared (the paper's layer shape)."""
    return Layer(0, 2048, 512, 256)


def test_moe_decode_m1(qwen_layer):
    L = qwen_layer
    g = synth.rng(20)
    x = synth.normal_f32(g, (1, L.H))
    ids, wts = synth.routing(g, 1, L.E, 8)
    out, h, hq, perm, count, ws = L.run(x, ids, wts, 8)
    st = L.check(x, ids, wts, 8, out, h, hq)
    assert st["pairs"] == 9
    # same workspace again: identical bytes
    out2, *_ = L.run(x, ids, wts, 8, ws=ws)
    assert np.array_equal(out, out2)


def test_moe_decode_m1_many_steps_one_workspace(qwen_layer):
    """Back-to-back single-token calls on one workspace with fresh routing,
    including skipped slots and a repeated expert: the in-kernel counters must
    return to zero after every call."""
    L = qwen_layer
    g = synth.rng(23)
    ws = w4.moe_workspace(1, L.H, L.I, L.E, 8)
    for step in range(6):
        x = synth.normal_f32(g, (1, L.H))
        ids, wts = synth.routing(g, 1, L.E, 8)
        if step == 2:
            ids[0, 3] = -1
        if step == 3:
            ids[0, 5] = ids[0, 1]
        if step == 4:
            ids[0, :] = -1
        out, h, hq, _, _, _ = L.run(x, ids, wts, 8, ws=ws)
        L.check(x, ids, wts, 8, out, h, hq)


def test_moe_decode_m1_wait_fallback(qwen_layer):
    """Force the bounded wait of the single-launch decode kernel to expire at
    once (poll bound 0 set from the host through w4a8_decode_wait_bound):
    every down-projection workgroup then computes its pair's h itself.  Same
    bytes as the normal path, and the counters still return to zero."""
    L = qwen_layer
    g = synth.rng(24)
    x = synth.normal_f32(g, (1, L.H))
    ids, wts = synth.routing(g, 1, L.E, 8)
    ws = w4.moe_workspace(1, L.H, L.I, L.E, 8)
    out, h, hq, *_ = L.run(x, ids, wts, 8, ws=ws)
    prev = w4.decode_wait_bound(0)
    try:
        out_fb, h_fb, hq_fb, *_ = L.run(x, ids, wts, 8, ws=ws)
    finally:
        assert w4.decode_wait_bound(prev) == 0
    assert np.array_equal(out, out_fb) and np.array_equal(hq, hq_fb)
    L.check(x, ids, wts, 8, out_fb, h_fb, hq_fb)
    x2 = synth.normal_f32(g, (1, L.H))
    ids2, wts2 = synth.routing(g, 1, L.E, 8)
    out2, h2, hq2, *_ = L.run(x2, ids2, wts2, 8, ws=ws)
    L.check(x2, ids2, wts2, 8, out2, h2, hq2)


def test_moe_workspace_reused_across_shapes(qwen_layer):
    """One workspace for a 32-token call with k = 4 (the grouped path writes
    its sort, tile and activation regions), then single-token calls with
    k = 8, whose hand-off region lies in the same workspace: each checked
    against the oracle (no stale hand-off word may be taken as this call's)."""
    L = qwen_layer
    g = synth.rng(27)
    ws = w4.moe_workspace(32, L.H, L.I, L.E, 8)
    x = synth.normal_f32(g, (32, L.H))
    ids, wts = synth.routing(g, 32, L.E, 4)
    out, h, hq, *_ = L.run(x, ids, wts, 4, ws=ws)
    L.check(x, ids, wts, 4, out, h, hq)
    for _ in range(3):
        x = synth.normal_f32(g, (1, L.H))
        ids, wts = synth.routing(g, 1, L.E, 8)
        out, h, hq, *_ = L.run(x, ids, wts, 8, ws=ws)
        L.check(x, ids, wts, 8, out, h, hq)


def test_moe_decode_m1_no_shared_small_shapes():
    """Single-token path at other shapes: H = 768 (three 8-block groups per
    row), I = 256, no shared expert, k = 3."""
    L = Layer(25, 768, 256, 6, shared=False)
    g = synth.rng(26)
    for _ in range(3):
        x = synth.normal_f32(g, (1, L.H))
        ids, wts = synth.routing(g, 1, L.E, 3)
        out, h, hq, *_ = L.run(x, ids, wts, 3)
        L.check(x, ids, wts, 3, out, h, hq)


def test_moe_decode_m32(qwen_layer):
    L = qwen_layer
    g = synth.rng(21)
    x = synth.normal_f32(g, (32, L.H))
    ids, wts = synth.routing(g, 32, L.E, 8)
    out, h, hq, perm, count, _ = L.run(x, ids, wts, 8)
    _check_route(ids, L.E, True, perm, count)
    L.check(x, ids, wts, 8, out, h, hq)


@pytest.mark.parametrize("E", [4, 128])
def test_moe_tile_kinds_above_128_tokens(E):
    """Above 128 tokens every expert group takes the MFMA tiles, its last
    tile by its rows: groups of 8 and 16 rows (16-row tiles, 16x16x32
    products), 17 rows (one 32-row half), 33 rows and the shared expert's
    136, checked token by token; the other slots skipped.  E = 4: so few
    tiles that the route cuts 32-row tiles; E = 128 (experts 4.. unused):
    64-row tiles, both halves for 33 rows."""
    L = Layer(7, 256, 256, E)
    g = synth.rng(31)
    T, k = 136, 2
    x = synth.normal_f32(g, (T, L.H))
    ids = np.full((T, k), -1, dtype=np.int32)
    ids[:8, 0] = 0                       # expert 0: 8 rows
    ids[8:24, 0] = 1                     # expert 1: 16 rows
    ids[24:40, 0] = 2                    # expert 2: 16 + 1 = 17 rows
    ids[:1, 1] = 2
    ids[1:34, 1] = 3                     # expert 3: 33 rows
    wts = g.random((T, k), dtype=np.float32)
    out, h, hq, perm, count, _ = L.run(x, ids, wts, k)
    assert count[:4].tolist() == [8, 16, 17, 33]
    _check_route(ids, L.E, True, perm, count)
    L.check(x, ids, wts, k, out, h, hq)


@pytest.mark.parametrize("E", [4, 128])
def test_moe_tiles_across_64_row_boundaries(E):
    """Groups of 64, 65, 97 and 30 rows plus the shared expert's 136, eight
    tokens with a skipped second slot.  E = 128 (experts 4.. unused): 64-row
    tiles -- one full tile, a full tile and a 1-row tile, a full tile and a
    33-row tile (second half in use), a 30-row half, two full tiles and an
    8-row tile; E = 4: the same groups in 32-row tiles."""
    L = Layer(7, 256, 256, E)
    g = synth.rng(33)
    T, k = 136, 2
    x = synth.normal_f32(g, (T, L.H))
    ids = np.full((T, k), -1, dtype=np.int32)
    ids[:64, 0] = 0
    ids[64:128, 0] = 1
    ids[128:, 0] = 3
    ids[:1, 1] = 1                       # expert 1: 65 rows
    ids[1:98, 1] = 2                     # expert 2: 97 rows
    ids[98:120, 1] = 3                   # expert 3: 8 + 22 = 30 rows
    wts = g.random((T, k), dtype=np.float32)
    out, h, hq, perm, count, _ = L.run(x, ids, wts, k)
    assert count[:4].tolist() == [64, 65, 97, 30]
    _check_route(ids, L.E, True, perm, count)
    L.check(x, ids, wts, k, out, h, hq)


@pytest.mark.parametrize("seed,H,I,E,shared,T,k", [
    (41, 768, 768, 5, True, 136, 2),     # three 8-block groups per row on both sides
    (42, 512, 256, 3, False, 136, 2),    # no shared expert; down K = 256 (one group)
    (43, 2560, 256, 2, True, 136, 1),    # K = 2560: ten staged groups for gate/up
])
def test_moe_mfma_path_shapes(seed, H, I, E, shared, T, k):
    """Shapes other than the paper's layer on the MFMA tiles (every group
    above 128 tokens)."""
    L = Layer(seed, H, I, E, shared=shared)
    g = synth.rng(seed + 100)
    x = synth.normal_f32(g, (T, L.H))
    ids, wts = synth.routing(g, T, L.E, k)
    out, h, hq, perm, count, _ = L.run(x, ids, wts, k)
    assert count.max() > 8
    _check_route(ids, L.E, shared, perm, count)
    L.check(x, ids, wts, k, out, h, hq)


def test_moe_route_4096_experts():
    """The largest expert count the library accepts: the route kernel's
    histogram then holds one segment per expert and the group counters reuse
    its space.  136 tokens: every group on the MFMA tiles, groups of one or
    two rows on 16-row tiles."""
    L = Layer(44, 256, 256, 4096)
    g = synth.rng(144)
    T, k = 136, 3
    x = synth.normal_f32(g, (T, L.H))
    ids, wts = synth.routing(g, T, L.E, k)
    ids[:40, 0] = 4095                   # one group of 40 rows
    ids[40:52, 1] = 17                   # one of 12 beside single rows
    out, h, hq, perm, count, _ = L.run(x, ids, wts, k)
    _check_route(ids, L.E, True, perm, count)
    L.check(x, ids, wts, k, out, h, hq)


@pytest.mark.parametrize("seed,E,T,k", [
    (45, 8, 100, 2),        # 200 pairs, one slice; 64 threads per expert sum the counts
    (46, 300, 129, 8),      # two threads per expert, two slices
    (47, 1000, 300, 8),     # one thread per expert (E not a power of two), three slices
    (48, 1024, 64, 8),      # the largest expert count of the split route
    (50, 256, 128, 8),      # exactly one full slice (1024 pairs): routed in the prep launch
    (49, 64, 2600, 8),      # 20800 pairs in 21 slices
])
def test_moe_split_route_shapes(seed, E, T, k):
    """The split route (per-slice ranks beside the quantization; a single
    slice finished in its own workgroup, several by one workgroup per slice
    placing its pairs and one writing the group lists) across expert counts
    and slice counts, with skipped and duplicate slots: the permutation and
    counts exact, every pair through the MoE check."""
    L = Layer(seed, 256, 256, E)
    g = synth.rng(seed + 200)
    x = synth.normal_f32(g, (T, L.H))
    ids, wts = synth.routing(g, T, L.E, k, bias_std=1.0)
    ids[1, 0] = -1                       # skipped slot
    ids[2, k - 1] = E                    # id >= E: skipped
    if k > 1:
        ids[3, 1] = ids[3, 0]            # duplicate expert in one token
    ids[min(T - 1, 70):, 0] = E - 1      # one long group (MFMA tiles above 128 tokens)
    out, h, hq, perm, count, _ = L.run(x, ids, wts, k)
    _check_route(ids, L.E, True, perm, count)
    ids_o = ids.copy(); ids_o[ids_o >= L.E] = -1
    L.check(x, ids_o, wts, k, out, h, hq)


@pytest.mark.parametrize("T", [100, 128])
def test_moe_mid_batch_on_the_valu_path(qwen_layer, T):
    """Up to 128 tokens every group takes the small-group VALU kernels in
    chunks of 8 rows, also groups of dozens of rows and the shared group of
    T rows (13 and 16 chunks), with biased routing: every token and pair
    through the MoE check."""
    L = qwen_layer
    g = synth.rng(23 + T)
    k = 8
    x = synth.normal_f32(g, (T, L.H))
    ids, wts = synth.routing(g, T, L.E, k, bias_std=1.0)
    out, h, hq, perm, count, _ = L.run(x, ids, wts, k)
    _check_route(ids, L.E, True, perm, count)
    assert count.max() > 16
    st = L.check(x, ids, wts, k, out, h, hq)
    assert st["pairs"] == T * (k + 1)


def test_moe_prefill_947_all_tokens(qwen_layer):
    """The 947-token prefill with biased routing (skewed expert load: empty
    experts, groups of a few rows on 16-row tiles, groups of hundreds of
    rows on 64-row tiles, the 947-row shared group): every token and every
    pair through the MoE check, and a second call bit-identical."""
    L = qwen_layer
    g = synth.rng(22)
    T, k = 947, 8
    x = synth.normal_f32(g, (T, L.H))
    ids, wts = synth.routing(g, T, L.E, k, bias_std=1.0)
    out, h, hq, perm, count, ws = L.run(x, ids, wts, k)
    _check_route(ids, L.E, True, perm, count)
    assert count.max() > 64 and (count[count > 0] <= 8).any()
    st = L.check(x, ids, wts, k, out, h, hq)
    assert st["pairs"] == T * (k + 1)
    out2, *_ = L.run(x, ids, wts, k, ws=ws)
    assert np.array_equal(out, out2)


def _first_experts(L, E):
    """A view of layer L restricted to its first E routed experts (the
    expert-major weight arrays cut after expert E - 1), shared expert kept."""
    V = Layer.__new__(Layer)
    V.H, V.I, V.E = L.H, L.I, E
    V.w_gu = L.w_gu.reshape(L.E, -1)[:E].reshape(-1)
    V.w_d = L.w_d.reshape(L.E, -1)[:E].reshape(-1)
    V.ws_gu, V.ws_d = L.ws_gu, L.ws_d
    V.d_gu, V.d_d = dev(V.w_gu), dev(V.w_d)
    V.d_sgu, V.d_sd = L.d_sgu, L.d_sd
    V.g = L.g
    return V


@pytest.mark.parametrize("T,bias", [(1, 0.0), (32, 0.0), (947, 1.0)])
@pytest.mark.parametrize("E,k", [(256, 4), (128, 8)])
def test_moe_full_shape_top4_and_128_experts(qwen_layer, T, bias, E, k):
    """The paper's two model variants at the full layer shape (H = 2048, I =
    512): top-4 of 256 routed experts, and 128 routed experts (the pruned
    model) at top-8, each at one token (the decode kernel), 32 tokens (the
    small-group kernels) and 947 tokens with skewed routing (small groups,
    MFMA tiles and the 947-row shared group); every token and pair through
    the MoE check, the routing permutation exact."""
    L = qwen_layer if E == qwen_layer.E else _first_experts(qwen_layer, E)
    g = synth.rng(900 + T + E + k)
    x = synth.normal_f32(g, (T, L.H))
    ids, wts = synth.routing(g, T, E, k, bias_std=bias)
    out, h, hq, perm, count, _ = L.run(x, ids, wts, k)
    if T > 1:
        _check_route(ids, E, True, perm, count)
    st = L.check(x, ids, wts, k, out, h, hq)
    assert st["pairs"] == T * (k + 1)


# ------------------------------------------------------------ RMSNorm + residual
@pytest.mark.parametrize("T,H,resid", [(1, 2048, True), (5, 256, False), (947, 2048, True), (3, 4100, True)])
def test_rmsnorm_residual_matches_oracle(T, H, resid):
    g = synth.rng(40 + T)
    x = synth.normal_f32(g, (T, H))
    y = synth.normal_f32(g, (T, H), 0.3) if resid else None
    gamma = (np.float32(1.0) + synth.normal_f32(g, (H,), 0.1)).astype(np.float32)
    xo_ref, xn_ref = oracle.rmsnorm_residual(x, y, gamma, eps=1e-6)
    xo, xn = w4.rmsnorm_residual(dev(x), None if y is None else dev(y), dev(gamma), eps=1e-6)
    assert np.array_equal(host(xo), xo_ref), "x + y must be one fp32 add"
    # fp32 sum of squares and three fp32 roundings per element
    err = np.abs(host(xn).astype(np.float64) - xn_ref)
    assert np.all(err <= 2e-6 * np.abs(xn_ref) + 1e-7 * np.abs(gamma).max())


def test_rmsnorm_residual_in_place_and_no_norm():
    g = synth.rng(47)
    x = synth.normal_f32(g, (4, 512))
    y = synth.normal_f32(g, (4, 512))
    gamma = np.ones(512, np.float32)
    xd = dev(x)
    xo, xn = w4.rmsnorm_residual(xd, dev(y), dev(gamma), x_out=xd)      # in place
    ref, xn_ref = oracle.rmsnorm_residual(x, y, gamma)
    assert np.array_equal(host(xd), ref)
    assert np.allclose(host(xn), xn_ref, rtol=2e-6, atol=1e-7)
    xo2, none = w4.rmsnorm_residual(dev(x), dev(y), None, want_norm=False)
    assert none is None and np.array_equal(host(xo2), ref)


# ------------------------------------------------------ pre-norm residual layer
@pytest.mark.parametrize("T,with_prev", [(1, True), (1, False), (6, True), (40, True)])
def test_moe_layer_residual_norm(qwen_layer, T, with_prev):
    """x_out = x + y_prev is one fp32 add, xn = RMSNorm(x_out) * gamma is within
    fp32 rounding of the oracle, Q8_0(xn) is bit-exact for the GPU's own xn,
    and the layer output is the MoE layer of that xn (T = 1: the norm inside
    the single decode launch; T > 1: the norm inside the quantizing
    workgroups of the prep launch, then the grouped path)."""
    L = qwen_layer
    g = synth.rng(60 + T)
    x = synth.normal_f32(g, (T, L.H))
    y_prev = synth.normal_f32(g, (T, L.H), 0.3) if with_prev else None
    gamma = (np.float32(1.0) + synth.normal_f32(g, (L.H,), 0.1)).astype(np.float32)
    ids, wts = synth.routing(g, T, L.E, 8)
    ws = w4.moe_workspace(T, L.H, L.I, L.E, 8)
    x_out, out = w4.moe_layer(dev(x), None if y_prev is None else dev(y_prev), dev(gamma),
                              dev(ids), dev(wts), L.d_gu, L.d_d, L.d_sgu, L.d_sd,
                              L.H, L.I, L.E, 8, ws)
    xo_ref, xn_ref = oracle.rmsnorm_residual(x, y_prev, gamma, eps=1e-6)
    assert np.array_equal(host(x_out), xo_ref)
    lay = w4.moe_workspace_layout(T, L.H, L.I, L.E, 8)
    wsn = host(ws)
    xn = wsn[lay["xn"]:lay["xn"] + T * L.H * 4].view(np.float32).reshape(T, L.H)
    err = np.abs(xn.astype(np.float64) - xn_ref)
    assert np.all(err <= 2e-6 * np.abs(xn_ref) + 1e-7 * np.abs(gamma).max())
    xq = wsn[lay["xq"]:lay["xq"] + T * (L.H // 32) * 34].reshape(T, -1)
    assert np.array_equal(xq, oracle.q8_0_quantize(xn)), "Q8_0 of the normalized row"
    P = T * 8 + T
    h = wsn[lay["h"]:lay["h"] + P * L.I * 4].view(np.float32).reshape(P, L.I)
    hq = wsn[lay["hq"]:lay["hq"] + P * (L.I // 32) * 34].reshape(P, -1)
    L.check(xn, ids, wts, 8, host(out), h, hq)


@pytest.mark.parametrize("H,T", [(4352, 5), (768, 21)])
def test_moe_layer_residual_norm_other_widths(H, T):
    """Rows wider than one quantizing workgroup (H = 4352: the norm in a
    launch of its own) and a width that leaves threads of the workgroup idle
    (H = 768: five rows per workgroup, 64 threads without a row)."""
    I, E, k = 256, 4, 2
    L = Layer(80 + H, H, I, E)
    g = synth.rng(81 + H)
    x = synth.normal_f32(g, (T, H))
    y_prev = synth.normal_f32(g, (T, H), 0.3)
    gamma = (np.float32(1.0) + synth.normal_f32(g, (H,), 0.1)).astype(np.float32)
    ids, wts = synth.routing(g, T, E, k)
    ws = w4.moe_workspace(T, H, I, E, k)
    x_out, out = w4.moe_layer(dev(x), dev(y_prev), dev(gamma), dev(ids), dev(wts), L.d_gu, L.d_d,
                              L.d_sgu, L.d_sd, H, I, E, k, ws)
    xo_ref, xn_ref = oracle.rmsnorm_residual(x, y_prev, gamma, eps=1e-6)
    assert np.array_equal(host(x_out), xo_ref)
    lay = w4.moe_workspace_layout(T, H, I, E, k)
    wsn = host(ws)
    xn = wsn[lay["xn"]:lay["xn"] + T * H * 4].view(np.float32).reshape(T, H)
    err = np.abs(xn.astype(np.float64) - xn_ref)
    assert np.all(err <= 2e-6 * np.abs(xn_ref) + 1e-7 * np.abs(gamma).max())
    xq = wsn[lay["xq"]:lay["xq"] + T * (H // 32) * 34].reshape(T, -1)
    assert np.array_equal(xq, oracle.q8_0_quantize(xn)), "Q8_0 of the normalized row"
    P = T * k + T
    h = wsn[lay["h"]:lay["h"] + P * I * 4].view(np.float32).reshape(P, I)
    hq = wsn[lay["hq"]:lay["hq"] + P * (I // 32) * 34].reshape(P, -1)
    L.check(xn, ids, wts, k, host(out), h, hq)


@pytest.mark.parametrize("T,gated", [(1, True), (1, False), (6, True), (40, True), (136, False)])
def test_moe_layer_routed(qwen_layer, T, gated):
    """Router in front of the residual layer: ids bit-exact with the oracle's
    top-k of the logits and weights within 4e-6; x_out, the normalized row
    and its Q8_0 as for moe_layer; the output through the MoE check, with the
    GPU's own routing weights for the routed slots (they are the layer's
    input) and the oracle's fp64 sigmoid of the gate for the shared expert
    (T = 1: the routing inside the single decode launch; T = 6 and 40: the
    VALU path; T = 136: the MFMA tiles)."""
    L = qwen_layer
    g = synth.rng(80 + T)
    x = synth.normal_f32(g, (T, L.H))
    y_prev = synth.normal_f32(g, (T, L.H), 0.3)
    gamma = (np.float32(1.0) + synth.normal_f32(g, (L.H,), 0.1)).astype(np.float32)
    logits = synth.normal_f32(g, (T, L.E))
    logits[:, :16] += np.float32(1.5)              # a few popular experts
    gate = synth.normal_f32(g, (T,), 2.0) if gated else None
    ws = w4.moe_workspace(T, L.H, L.I, L.E, 8)
    x_out, out, ids_d, w_d = w4.moe_layer_routed(
        dev(x), dev(y_prev), dev(gamma), dev(logits), L.d_gu, L.d_d, L.d_sgu, L.d_sd,
        L.H, L.I, L.E, 8, ws, shared_gate=dev(gate) if gated else None)
    ids, wts = host(ids_d), host(w_d)
    ids_r, w_r = oracle.router_topk(logits, 8)
    assert np.array_equal(ids, ids_r)
    assert np.all(np.abs(wts.astype(np.float64) - w_r) <= 4e-6 * w_r)
    xo_ref, xn_ref = oracle.rmsnorm_residual(x, y_prev, gamma, eps=1e-6)
    assert np.array_equal(host(x_out), xo_ref)
    lay = w4.moe_workspace_layout(T, L.H, L.I, L.E, 8)
    wsn = host(ws)
    xn = wsn[lay["xn"]:lay["xn"] + T * L.H * 4].view(np.float32).reshape(T, L.H)
    err = np.abs(xn.astype(np.float64) - xn_ref)
    assert np.all(err <= 2e-6 * np.abs(xn_ref) + 1e-7 * np.abs(gamma).max())
    P = T * 8 + T
    h = wsn[lay["h"]:lay["h"] + P * L.I * 4].view(np.float32).reshape(P, L.I)
    hq = wsn[lay["hq"]:lay["hq"] + P * (L.I // 32) * 34].reshape(P, -1)
    sw = 1.0 / (1.0 + np.exp(-gate.astype(np.float64))) if gated else None
    L.check(xn, ids, wts, 8, host(out), h, hq, shared_w=sw)


@pytest.mark.parametrize("E,k,ties,gated", [(256, 8, True, True), (300, 8, False, False),
                                             (512, 32, True, True), (8, 8, True, False)])
def test_routed_decode_matches_router_kernel(E, k, ties, gated):
    """T = 1: the top-k taken inside the single-token launch gives the router
    kernel's ids and weights bit for bit (the same wave top-k on both), with
    equal logits, with 256 < E <= 512 (eight logits per lane) and with k = E;
    ids also against the oracle, the layer output through the MoE check."""
    L = Layer(90 + E, 256, 256, E)
    g = synth.rng(91 + E + k)
    x = synth.normal_f32(g, (1, L.H))
    y_prev = synth.normal_f32(g, (1, L.H), 0.3)
    gamma = np.ones(L.H, np.float32)
    logits = synth.normal_f32(g, (1, E))
    if ties:
        logits = (np.round(logits * 2.0) / 2.0).astype(np.float32)
    gate = synth.normal_f32(g, (1,), 2.0) if gated else None
    ws = w4.moe_workspace(1, L.H, L.I, E, k)
    x_out, out, ids_d, w_d = w4.moe_layer_routed(
        dev(x), dev(y_prev), dev(gamma), dev(logits), L.d_gu, L.d_d, L.d_sgu, L.d_sd,
        L.H, L.I, E, k, ws, shared_gate=dev(gate) if gated else None)
    ids_k, w_k = w4.router_topk(dev(logits), k)
    ids, wts = host(ids_d), host(w_d)
    assert np.array_equal(ids, host(ids_k))
    assert np.array_equal(wts.view(np.uint32), host(w_k).view(np.uint32))
    assert np.array_equal(ids, oracle.router_topk(logits, k)[0])
    lay = w4.moe_workspace_layout(1, L.H, L.I, E, k)
    wsn = host(ws)
    xn = wsn[lay["xn"]:lay["xn"] + L.H * 4].view(np.float32).reshape(1, L.H)
    P = k + 1
    h = wsn[lay["h"]:lay["h"] + P * L.I * 4].view(np.float32).reshape(P, L.I)
    hq = wsn[lay["hq"]:lay["hq"] + P * (L.I // 32) * 34].reshape(P, -1)
    sw = 1.0 / (1.0 + np.exp(-gate.astype(np.float64))) if gated else None
    L.check(xn, ids, wts, k, host(out), h, hq, shared_w=sw)


# ------------------------------------------------------------ router top-k
@pytest.mark.parametrize("T,E,k", [(1, 256, 8), (947, 256, 8), (5, 7, 7), (33, 4096, 32),
                                   (64, 64, 1), (3, 130, 32), (2, 10, 4)])
def test_router_topk_matches_oracle(T, E, k):
    """ids bit-exact (the selection compares the fp32 logits on both sides);
    weights within 4e-6 relative: fp32 rounding of l - l_max (|l - l_max| of
    at most ~10 here, 2^-24 each), of expf (2 ulp), of the k-term sum and of
    the division."""
    g = synth.rng(70 + T + E + k)
    logits = synth.normal_f32(g, (T, E))
    logits[0] = np.round(logits[0] * 2.0) / 2.0            # many equal logits
    if E == 10:
        logits[:] = 0.0                                    # all equal
    ids, w = w4.router_topk(dev(logits), k)
    ids_r, w_r = oracle.router_topk(logits, k)
    assert np.array_equal(host(ids), ids_r)
    err = np.abs(host(w).astype(np.float64) - w_r)
    assert np.all(err <= 4e-6 * w_r), f"max rel err {np.max(err / w_r):.3g}"


def test_router_output_feeds_the_layer(small_layer):
    """The router's ids and weights drive a 40-token layer as given."""
    L = small_layer
    g = synth.rng(77)
    T, k = 40, 2
    x = synth.normal_f32(g, (T, L.H))
    logits = synth.normal_f32(g, (T, L.E))
    ids_d, w_d = w4.router_topk(dev(logits), k)
    ids, wts = host(ids_d), host(w_d)
    ids_r, _ = oracle.router_topk(logits, k)
    assert np.array_equal(ids, ids_r)
    out, h, hq, perm, count, _ = L.run(x, ids, wts, k)
    _check_route(ids, L.E, True, perm, count)
    L.check(x, ids, wts, k, out, h, hq)
