"""Device path (libcats through the C ABI) against the CPU oracle.

Same seeded inputs on both sides; the oracle is the fp32 build.  Bars:
  - active sets identical except neurons with ||v| - t| <= 1e-3 t
  - y within 2e-2 * ||y_oracle||_inf (measured errors are far smaller)
  - index work (pack, threshold selection) bit-exact
"""
import os

import numpy as np
import pytest
import torch

import paper_2404_08763_amd as P
from paper_2404_08763_amd import workloads as W

from gpu_util import Y_TOL, band_ok, check_forward, device_layer, h_bound, host_f32, quantile_t, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a device"
    return torch.device("cuda:0")


def test_single_hip_runtime(dev):
    """libcats binds to the HIP runtime torch loaded (one copy in the process)."""
    P.raw()
    torch.zeros(1, device=dev)
    maps = open("/proc/self/maps").read().splitlines()
    paths = {ln.split()[-1] for ln in maps if "libamdhip64" in ln}
    assert len(paths) == 1, paths
    assert any(P.lib_path() in ln for ln in maps)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("shape", [(37, 53), (4096, 688), (1, 9), (256, 688)])
def test_pack_bit_exact(dev, dtype, shape):
    say("pack", dtype, shape)
    g = torch.Generator().manual_seed(5)
    w = torch.randn(shape, generator=g).to(dtype)
    out = P.pack_weights(w.to(dev)).cpu()
    ref = w.t().contiguous()
    assert torch.equal(out.view(torch.int16 if dtype == torch.bfloat16 else torch.int32),
                       ref.view(torch.int16 if dtype == torch.bfloat16 else torch.int32))


# ---------------------------------------------------------------- C1 (tiny)
@pytest.fixture(scope="module")
def c1(dev, oracle32):
    c = W.CONFIGS["C1"]
    wg, wu, wd = W.weights(c.d, c.m, c.wdtype)
    layer = device_layer(wg, wu, wd)
    hw = host_f32(wg, wu, wd)
    xcal = W.calib_vectors(c)
    acts = oracle32.calib_acts(xcal.numpy(), hw[0])
    t = oracle32.threshold(acts, 0.5)
    return c, layer, hw, xcal, acts, t


def test_c1_forward_all_vectors(c1, oracle32):
    c, layer, hw, _, _, t = c1
    xs = W.decode_vectors(c)
    ws = P.workspace(c.d, c.m, 1)
    flips = 0
    for i in range(c.n_decode):
        say("C1 forward vector", i, "t", t)
        x = xs[i : i + 1].contiguous()
        y, aux = P.mlp_forward(layer, x.cuda(), t, ws=ws, aux=True)
        ref = oracle32.cats_mlp(x.numpy(), *hw, t=t)
        ref_all = oracle32.cats_mlp(x.numpy(), *hw, t=0.0)
        flips += check_forward(y, aux, ref, t, 1, f"C1[{i}]", ref_all=ref_all, w_down=hw[2])["band_flips"]
    assert flips <= 3


def test_c1_dense_and_t0(c1, oracle32):
    c, layer, hw, _, _, _ = c1
    x = W.decode_vectors(c, 4)
    say("C1 dense B=4")
    yd = P.mlp_dense(layer, x.cuda())
    ref = oracle32.cats_mlp(x.numpy(), *hw, t=0.0, dense=True)
    check_forward(yd, None, ref, 0.0, 4, "C1 dense")
    say("C1 forward t=0 B=4")
    y0 = P.mlp_forward(layer, x.cuda(), 0.0)
    assert torch.equal(y0.view(torch.int32), yd.view(torch.int32)), "t=0 must equal dense bit for bit"


def test_c1_calibration(c1, oracle32):
    c, layer, hw, xcal, acts_o, t_o = c1
    say("C1 calibrate")
    xg = xcal.cuda()
    acts = P.calib_activations(layer, xg)
    a = acts.cpu().double().numpy()
    assert np.abs(a - acts_o).max() <= 1e-5 * acts_o.max()
    t = P.calibrate_threshold(layer, xg, 0.5)
    assert abs(t - t_o) <= 1e-3 * t_o, (t, t_o)
    # the rank invariant of Eq. 3 on the device's own activations
    s = np.sort(a.ravel())
    n = s.size
    r = int(np.ceil(0.5 * n - 1e-6))
    assert t == np.float32(s[r - 1])
    assert int(np.sum(s < t)) <= r - 1 < 0.5 * n <= r <= int(np.sum(s <= t))


# ------------------------------------------- small bf16 shapes, ragged tails
@pytest.mark.parametrize("d,m", [(1032, 693), (512, 1000), (8, 7), (4096, 97), (5120, 300), (8192, 64)])
def test_bf16_ragged_shapes(dev, oracle32, d, m):
    c = W.shrink(W.CONFIGS["C2"], d, m)
    wg, wu, wd = W.weights(d, m, torch.bfloat16, layer=3)
    layer = device_layer(wg, wu, wd)
    hw = host_f32(wg, wu, wd)
    x = W.decode_vectors(c, 3)
    all0 = [oracle32.cats_mlp(x[b : b + 1].numpy(), *hw, t=0.0) for b in range(3)]
    v0 = np.concatenate([r["v"] for r in all0], axis=0)
    for k in (0.5, 0.9):
        t = quantile_t(np.abs(v0), k)
        say("ragged", d, m, "k", k, "t", t)
        for b in range(3):
            xb = x[b : b + 1].contiguous()
            y, aux = P.mlp_forward(layer, xb.cuda(), t, aux=True)
            ref = oracle32.cats_mlp(xb.numpy(), *hw, t=t)
            check_forward(y, aux, ref, t, 1, f"d{d} m{m} k{k} b{b}", ref_all=all0[b], w_down=hw[2])


@pytest.mark.parametrize("dtype,d,m,B", [(torch.bfloat16, 8192, 2600, 1), (torch.bfloat16, 8192, 2600, 3),
                                         (torch.float32, 4096, 1500, 1), (torch.float32, 4096, 1500, 2)])
def test_wide_rows(dev, oracle32, dtype, d, m, B):
    """Rows of 16 chunks per lane (bf16 d = 8192, fp32 d = 4096): the fused
    kernel runs four waves per block there, each wave holding its row
    buffers in the whole register file of a SIMD; about 10 neurons per block."""
    c = W.shrink(W.CONFIGS["C3"], d, m)
    wg, wu, wd = W.weights(d, m, dtype, layer=8)
    layer = device_layer(wg, wu, wd)
    hw = host_f32(wg, wu, wd)
    x = W.decode_vectors(c, B)
    ref_all = oracle32.cats_mlp(x.numpy(), *hw, t=0.0)
    for k in (0.0, 0.6):
        t = quantile_t(np.abs(ref_all["v"]), k) if k > 0 else 0.0
        say("wide rows", dtype, d, m, "B", B, "k", k)
        y, aux = P.mlp_forward(layer, x.cuda(), t, aux=True)
        ref = ref_all if k == 0 else oracle32.cats_mlp(x.numpy(), *hw, t=t)
        check_forward(y, aux, ref, t, B, f"wide {dtype} d{d} B{B} k{k}", ref_all=ref_all, w_down=hw[2])


@pytest.mark.parametrize("B", [2, 3, 4, 8, 16])
def test_batch_rows_have_their_own_masks(dev, oracle32, B):
    d, m = 1024, 1500
    c = W.shrink(W.CONFIGS["C3"], d, m)
    wg, wu, wd = W.weights(d, m, torch.bfloat16, layer=4)
    layer = device_layer(wg, wu, wd)
    hw = host_f32(wg, wu, wd)
    x = W.decode_vectors(c, B)
    ref_all = oracle32.cats_mlp(x.numpy(), *hw, t=0.0)
    t = quantile_t(np.abs(ref_all["v"]), 0.7)
    res = torch.randn((B, d), generator=torch.Generator().manual_seed(9))
    say("batch", B, "t", t)
    y, aux = P.mlp_forward(layer, x.cuda(), t, residual=res.cuda(), aux=True)
    ref = oracle32.cats_mlp(x.numpy(), *hw, t=t, residual=res.numpy())
    check_forward(y, aux, ref, t, B, f"B{B}", ref_all=ref_all, w_down=hw[2],
                  h_abs=h_bound(x.numpy(), hw[1], ref_all["v"]))
    # rows differ in their masks (contextual sparsity)
    cnt = aux["cnt"].cpu().numpy()
    assert len(set(cnt.tolist())) > 1 or B == 1
    # each row agrees with its own batch-1 call: the same active set outside
    # the band, y within the bar (from 5 rows on, bf16 weights take the
    # matrix-core path, whose x carries 16 of its 24 mantissa bits, so a
    # neuron in the band may flip between the two calls)
    for b in range(B):
        yb, auxb = P.mlp_forward(layer, x[b : b + 1].cuda(), t, residual=res[b : b + 1].cuda(), aux=True)
        scale = float(y[b].abs().max())
        assert float((yb[0] - y[b]).abs().max()) <= Y_TOL * scale
        n1, nb_ = int(auxb["cnt"][0]), int(aux["cnt"][b])
        bad, _ = band_ok(auxb["idx"][0, :n1].cpu().numpy(), aux["idx"][b, :nb_].cpu().numpy(),
                         np.abs(ref_all["v"][b]), t)
        assert not bad, (b, bad[:5])


# ------------------------------------------------ batched (matrix-core) path
# bf16 weights, 5..16 rows and d of 512, 1024, 2048, 3072, 4096 or 5120
@pytest.mark.parametrize("d,m,B", [(512, 7, 5), (512, 300, 8), (1024, 693, 16), (1024, 693, 6), (3072, 500, 7),
                                   (4096, 1100, 16), (2048, 4111, 12), (5120, 700, 16), (5120, 2063, 5)])
def test_batched_path_vs_oracle(dev, oracle32, d, m, B):
    c = W.shrink(W.CONFIGS["C3"], d, m)
    wg, wu, wd = W.weights(d, m, torch.bfloat16, layer=6)
    layer = device_layer(wg, wu, wd)
    hw = host_f32(wg, wu, wd)
    x = W.decode_vectors(c, B)
    ref_all = oracle32.cats_mlp(x.numpy(), *hw, t=0.0)
    res = torch.randn((B, d), generator=torch.Generator().manual_seed(10))
    ws = P.workspace(d, m, B)
    for k in (0.0, 0.5, 0.9):
        t = quantile_t(np.abs(ref_all["v"]), k) if k > 0 else 0.0
        say("batched path d", d, "m", m, "B", B, "k", k, "t", t)
        y, aux = P.mlp_forward(layer, x.cuda(), t, residual=res.cuda(), ws=ws, aux=True)
        ref = ref_all if k == 0 else oracle32.cats_mlp(x.numpy(), *hw, t=t)
        ref = dict(ref)
        ref["y"] = ref["y"] + res.numpy().astype(np.float64)
        check_forward(y, aux, ref, t, B, f"batched d{d} m{m} B{B} k{k}", ref_all=ref_all, w_down=hw[2],
                      h_abs=h_bound(x.numpy(), hw[1], ref_all["v"]))
        y2 = P.mlp_forward(layer, x.cuda(), t, residual=res.cuda(), ws=ws)
        assert torch.equal(y.view(torch.int32), y2.view(torch.int32)), "aux outputs changed y"
    say("batched dense d", d, "B", B)
    yd = P.mlp_dense(layer, x.cuda(), ws=ws)
    check_forward(yd, None, oracle32.cats_mlp(x.numpy(), *hw, t=0.0, dense=True), 0.0, B, "batched dense")
    say("batched t=inf d", d, "B", B)
    yi = P.mlp_forward(layer, x.cuda(), float("inf"), residual=res.cuda(), ws=ws)
    assert torch.equal(yi.cpu(), res)


@pytest.mark.parametrize("name", ["C2", "C4"])
def test_batched_full_size(dev, oracle32, name):
    """Llama2-7B- and Llama2-13B-shaped blocks at 16 rows (the batched
    path), k = 0.5 and 0.7."""
    c = W.CONFIGS[name]
    wg, wu, wd = W.weights(c.d, c.m, c.wdtype)
    layer = device_layer(wg, wu, wd)
    hw = host_f32(wg, wu, wd)
    B = 16
    x = W.decode_vectors(c, B)
    ref_all = oracle32.cats_mlp(x.numpy(), *hw, t=0.0)
    ws = P.workspace(c.d, c.m, B)
    for k in (0.5, 0.7):
        t = quantile_t(np.abs(ref_all["v"]), k)
        say(name, "batched B16 k", k, "t", t)
        y, aux = P.mlp_forward(layer, x.cuda(), t, ws=ws, aux=True)
        ref = oracle32.cats_mlp(x.numpy(), *hw, t=t)
        r = check_forward(y, aux, ref, t, B, f"{name} B16 k{k}", ref_all=ref_all, w_down=hw[2],
                          h_abs=h_bound(x.numpy(), hw[1], ref_all["v"]))
        print(f"[batched] {name} B16 k{k}: y err {r['y_err']:.3e} (reconciled {r['y_err_reconciled']:.3e}) "
              f"of {r['y_scale']:.3e}, {r['band_flips']} band flips")
        y2 = P.mlp_forward(layer, x.cuda(), t, ws=ws)
        assert torch.equal(y.view(torch.int32), y2.view(torch.int32))


# ------------------------------------------------------ edge cases (C1 size)
def test_edges(c1, oracle32):
    c, layer, hw, _, _, _ = c1
    x = W.decode_vectors(c, 1)
    xg = x.cuda()
    res = torch.randn((1, c.d), generator=torch.Generator().manual_seed(2)).cuda()
    say("edges: t=inf")
    y, aux = P.mlp_forward(layer, xg, float("inf"), aux=True)
    assert int(aux["cnt"][0]) == 0
    assert torch.all(y == 0) and not torch.any(torch.signbit(y))
    y = P.mlp_forward(layer, xg, float("inf"), residual=res)
    assert torch.equal(y, res)
    say("edges: t=0 all active")
    y, aux = P.mlp_forward(layer, xg, 0.0, aux=True)
    assert int(aux["cnt"][0]) == c.m
    assert torch.equal(aux["idx"][0].cpu(), torch.arange(c.m, dtype=torch.int32))
    say("edges: one active neuron")
    v = oracle32.cats_mlp(x.numpy(), *hw, t=0.0)["v"][0]
    order = np.argsort(np.abs(v))
    t = float(0.5 * (abs(v[order[-1]]) + abs(v[order[-2]])))
    y, aux = P.mlp_forward(layer, xg, t, aux=True)
    assert int(aux["cnt"][0]) == 1 and int(aux["idx"][0, 0]) == int(order[-1])
    j = int(order[-1])
    h = aux["h"][0, 0].cpu()
    expect = h * torch.from_numpy(hw[2][j])  # fp32 product, rounded once
    assert torch.equal(y[0].cpu(), expect)


def test_determinism_and_aux_invariance(c1):
    c, layer, hw, _, _, t = c1
    x = W.decode_vectors(c, 8).cuda()
    say("determinism")
    y1, a1 = P.mlp_forward(layer, x, t, aux=True)
    y2, a2 = P.mlp_forward(layer, x, t, aux=True)
    y3 = P.mlp_forward(layer, x, t)
    assert torch.equal(y1.view(torch.int32), y2.view(torch.int32))
    assert torch.equal(y1.view(torch.int32), y3.view(torch.int32))
    for k in ("cnt", "idx", "v", "h"):
        if k == "cnt":
            assert torch.equal(a1[k], a2[k])
        else:
            for b in range(8):
                n = int(a1["cnt"][b])
                assert torch.equal(a1[k][b, :n], a2[k][b, :n])


def test_shared_workspace_across_shapes(dev, oracle32):
    """One workspace, filled with garbage first, serves calls of different
    shapes and batch sizes in a row (nothing a call needs is left over from
    the previous one)."""
    shapes = [(4096, 11008, 1), (256, 688, 3), (1032, 7, 2), (5120, 300, 4), (4096, 11008, 1)]
    nbytes = max(P.workspace_bytes(d, m, B, 0) for d, m, B in shapes)
    ws = torch.full((nbytes,), 0xAB, dtype=torch.uint8, device=dev)
    for i, (d, m, B) in enumerate(shapes):
        say("shared workspace", i, d, m, B)
        g = torch.Generator().manual_seed(300 + i)
        wg, wu, wd = [(torch.randn(sh, generator=g) * 0.02).to(torch.bfloat16)
                      for sh in ((d, m), (d, m), (m, d))]
        x = torch.randn((B, d), generator=g)
        layer = device_layer(wg, wu, wd)
        hw = host_f32(wg, wu, wd)
        ref_all = oracle32.cats_mlp(x.numpy(), *hw, t=0.0)
        t = quantile_t(np.abs(ref_all["v"]), 0.6)
        ref = oracle32.cats_mlp(x.numpy(), *hw, t=t)
        ys = [P.mlp_forward(layer, x.cuda(), t, ws=ws) for _ in range(3)]
        for y in ys[1:]:
            assert torch.equal(ys[0].view(torch.int32), y.view(torch.int32))
        check_forward(ys[0], None, ref, t, B, f"shared ws {d}x{m} B={B}")


def test_rmsnorm(dev, oracle32):
    for B, d in ((1, 4096), (3, 5120), (2, 7)):
        say("rmsnorm", B, d)
        x = torch.randn((B, d), generator=torch.Generator().manual_seed(d)) * 3
        y = P.rmsnorm(x.cuda(), 1e-5).cpu().double().numpy()
        ref = oracle32.rmsnorm(x.numpy(), 1e-5)
        assert np.abs(y - ref).max() <= 2e-6 * np.abs(ref).max()


def test_threshold_from_acts_bit_exact(dev, oracle32):
    g = torch.Generator().manual_seed(31)
    for n in (1, 7, 1000, 1 << 20, 3_000_001):
        a = torch.randn(n, generator=g)
        if n > 10:
            a[::13] = a[5]
            a[1::17] = -a[9]
        ag = a.cuda()
        for k in (0.0, 1e-6, 0.3, 0.5, 0.7, 0.9, 1.0):
            say("threshold n", n, "k", k)
            t = P.threshold_from_acts(ag, k)
            to = oracle32.threshold(a.double().numpy(), k)
            assert np.float32(t) == np.float32(to), (n, k, t, to)


# --------------------------------------- full-size shapes (sampled oracle)
@pytest.fixture(scope="module")
def big(dev):
    cache = {}

    def get(name):
        if name not in cache:
            cache.clear()
            c = W.CONFIGS[name]
            wg, wu, wd = W.weights(c.d, c.m, c.wdtype)
            cache[name] = (c, device_layer(wg, wu, wd), host_f32(wg, wu, wd))
        return cache[name]

    return get


@pytest.mark.parametrize("name,ks", [("C2", (0.5, 0.7, 0.9)), ("C3", (0.0, 0.3, 0.5, 0.7, 0.9))])
def test_full_size_forward(big, oracle32, name, ks):
    c, layer, hw = big(name)
    x = W.decode_vectors(c, 2)
    ws = P.workspace(c.d, c.m, 1)
    refs0 = [oracle32.cats_mlp(x[i : i + 1].numpy(), *hw, t=0.0) for i in range(2)]
    vall = np.concatenate([r["v"] for r in refs0], axis=0)
    for k in ks:
        t = quantile_t(np.abs(vall), k) if k > 0 else 0.0
        for i in range(2):
            say(name, "full-size forward k", k, "token", i, "t", t)
            xi = x[i : i + 1].contiguous()
            y, aux = P.mlp_forward(layer, xi.cuda(), t, ws=ws, aux=True)
            ref = refs0[i] if k == 0 else oracle32.cats_mlp(xi.numpy(), *hw, t=t)
            check_forward(y, aux, ref, t, 1, f"{name} k{k} tok{i}", ref_all=refs0[i], w_down=hw[2])
            y_noaux = P.mlp_forward(layer, xi.cuda(), t, ws=ws)  # the benchmark's configuration
            assert torch.equal(y.view(torch.int32), y_noaux.view(torch.int32))


@pytest.mark.parametrize("n", [4, 8])
def test_neuron_shard(big, oracle32, n):
    """One GPU's share of the C2 block split by neuron over n GPUs (its first
    m / n rows of all three neuron-major matrices), the shape the benchmark's
    shard figures run: at one row each wave owns two or three neurons."""
    c, layer, hw = big("C2")
    ms = c.m // n
    shard = P.Layer(layer.w_gate_t[:ms].contiguous(), layer.w_up_t[:ms].contiguous(),
                    layer.w_down[:ms].contiguous())
    hws = [np.ascontiguousarray(hw[0][:, :ms]), np.ascontiguousarray(hw[1][:, :ms]),
           np.ascontiguousarray(hw[2][:ms])]
    for B in (1, 3):
        x = W.decode_vectors(c, B).numpy()
        ref_all = oracle32.cats_mlp(x, *hws, t=0.0)
        t = quantile_t(np.abs(ref_all["v"]), 0.5)
        say("C2 shard 1 /", n, "B", B, "t", t)
        y, aux = P.mlp_forward(shard, torch.from_numpy(x).cuda(), t, aux=True)
        ref = oracle32.cats_mlp(x, *hws, t=t)
        check_forward(y, aux, ref, t, B, f"C2 shard 1/{n} B{B}", ref_all=ref_all, w_down=hws[2])


def test_full_size_dense(big, oracle32):
    c, layer, hw = big("C2")
    x = W.decode_vectors(c, 1)
    say("C2 dense")
    y = P.mlp_dense(layer, x.cuda())
    ref = oracle32.cats_mlp(x.numpy(), *hw, t=0.0, dense=True)
    check_forward(y, None, ref, 0.0, 1, "C2 dense")


def test_full_size_calibration_sampled(big, oracle32):
    c, layer, hw = big("C2")
    N = 256
    xcal = W.calib_vectors(c, N)
    say("C2 calibration activations N", N)
    acts = P.calib_activations(layer, xcal.cuda()).cpu().double().numpy()
    rng = np.random.default_rng(3)
    pairs = np.stack([rng.integers(0, N, 3000), rng.integers(0, c.m, 3000)], axis=1)
    ref = oracle32.calib_acts_at(xcal.numpy(), hw[0], pairs)
    got = acts[pairs[:, 0], pairs[:, 1]]
    assert np.abs(got - ref).max() <= 1e-5 * max(1.0, ref.max())
    for k in (0.5, 0.7, 0.9):
        say("C2 calibrate k", k)
        t = P.calibrate_threshold(layer, xcal.cuda(), k)
        s = np.sort(acts.ravel())
        n = s.size
        r = int(np.ceil(k * n - 1e-6))
        assert t == np.float32(s[r - 1])  # exact order statistic of the device's activations
        to = oracle32.threshold(acts, k)
        assert t == np.float32(to)
