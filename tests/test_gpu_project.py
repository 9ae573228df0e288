"""GPU parity of the fused projection (Sec. 3.1 Eq. (5)) against the float64 oracle.

Every case runs the HIP kernels through the C ABI and compares each example's
k_out x k_in gradient with the oracle's on the same input bytes.  Tolerances:
1e-4 normwise for fp32 inputs and 2e-2 for bf16 inputs (fp32 accumulation);
fp32 outputs of bf16 inputs are also held to 1e-3, what fp32 accumulation of
exact bf16 products leaves.
"""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

CASES = {
    # name: (dtype, B, T, n_in, n_out, k_in, k_out, x_std, dy_std, ragged, out_dtype)
    "tiny_f32": ("f32", 4, 16, 64, 64, 8, 8, 1.0, 1e-2, False, "f32"),
    "asym_bf16_ragged": ("bf16", 5, 150, 200, 328, 12, 20, 1.0, 0.5, True, "f32"),
    "asym_bf16_out_bf16": ("bf16", 5, 150, 200, 328, 12, 20, 1.0, 0.5, True, "bf16"),
    "f32_ragged_kt2": ("f32", 3, 77, 96, 52, 24, 7, 1.0, 1.0, True, "f32"),
    "k64_bf16": ("bf16", 3, 130, 512, 1024, 64, 64, 1.0, 1e-4, True, "f32"),
    "k128_bf16": ("bf16", 2, 70, 256, 136, 128, 100, 1.0, 1.0, True, "f32"),
    "gpt2_qkv": ("bf16", 3, 200, 768, 2304, 16, 16, 1.0, 1e-3, True, "bf16"),
    "llama_gate": ("bf16", 2, 96, 4096, 14336, 16, 16, 1.0, 1e-4, True, "bf16"),
    "llama_down_k64": ("bf16", 2, 65, 14336, 4096, 64, 64, 1.0, 1e-4, False, "f32"),
    # layers wider than one contraction chunk at k > 32 (chunks of 14,336 columns): the chunk
    # partials of several slots summed per tile, and P read from each chunk's column offset;
    # k = 64 takes the LDS-DMA path, k = 128 the register path
    "wide_in_k64_ragged": ("bf16", 3, 90, 16384, 1024, 64, 64, 1.0, 1e-3, True, "f32"),
    "wide_out_k128_ragged": ("bf16", 3, 70, 512, 28672, 128, 96, 1.0, 1e-3, True, "f32"),
    # and at k <= 32: an unpaired stream item per chunk (k = 16, bf16), the per-wave chunk
    # kernel (k = 16, fp32 inputs) and tile groups (k = 32)
    "wide_out_k16_ragged": ("bf16", 3, 90, 1024, 16384, 16, 16, 1.0, 1e-3, True, "bf16"),
    "wide_in_k16_f32": ("f32", 2, 40, 20000, 64, 16, 16, 1.0, 1e-2, True, "f32"),
    "wide_in_k32_ragged": ("bf16", 2, 70, 15000, 512, 32, 32, 1.0, 1e-3, True, "f32"),
}


def _inputs(name, seed=0):
    dt, B, T, n_in, n_out, k_in, k_out, xs, dys, ragged, _ = CASES[name]
    lens = None
    if ragged:
        lens = W.lengths(W.rng(seed, 7, B), B, 0, T)
        lens[0] = T
        if B > 2:
            lens[1] = 0
    return W.layer_inputs(seed, sorted(CASES).index(name), B, T, n_in, n_out, k_in, k_out, xs, dys, dt, lens)


def _run(d, out_dtype, g_ld=None, poison=False):
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host
    x, dy = d["x"].copy(), d["dy"].copy()
    if poison and d["mask"] is not None:
        m = d["mask"] == 0
        if x.dtype == np.uint16:
            x[m] = 0x7FC0      # NaN
            dy[m] = 0xFF80     # -Inf
        else:
            x[m] = np.nan
            dy[m] = np.inf
    B = x.shape[0]
    D = d["p_in"].shape[0] * d["p_out"].shape[0]
    tdt = torch.float32 if out_dtype == "f32" else torch.bfloat16
    store = torch.full((B, g_ld or D), 7.0, dtype=tdt, device="cuda")
    g = store[:, :D]
    P.logra_project_layer(dev(x), dev(dy), dev(d["p_in"]), dev(d["p_out"]), g,
                          mask=None if d["mask"] is None else dev(d["mask"]))
    torch.cuda.synchronize()
    return host(store)


@pytest.mark.parametrize("name", sorted(CASES))
def test_project_parity(name):
    from gpu_util import f64, rowwise_normwise, say
    say(f"[project parity] case={name}")
    d = _inputs(name)
    out_dtype = CASES[name][-1]
    got = _run(d, out_dtype)
    want = oracle.project_factored(d["x"], d["dy"], d["p_in"], d["p_out"], d["mask"])
    err = rowwise_normwise(got, want)
    tol = 1e-4 if CASES[name][0] == "f32" else 2e-2
    say(f"  normwise err {err:.3e} (tol {tol})")
    assert err <= tol
    if out_dtype == "f32" and CASES[name][0] == "bf16":
        assert err <= 1e-3
    if d["mask"] is not None:
        empty = d["mask"].sum(1) == 0
        assert np.all(f64(got)[empty] == 0.0)


def test_project_integer_exact():
    """Small-integer inputs make every product and sum exact in fp32: the GPU
    result must equal the oracle bit for bit (catches any index/layout slip)."""
    from gpu_util import say
    say("[project exact] integer inputs")
    g = W.rng(3, 11)
    B, T, n_in, n_out, k_in, k_out = 3, 100, 64, 48, 8, 16
    d = {"x": W.integer_array(g, (B, T, n_in), -1, 1, "bf16", 0.5),
         "dy": W.integer_array(g, (B, T, n_out), -1, 1, "bf16", 0.5),
         "p_in": W.integer_array(g, (k_in, n_in), -1, 1, "bf16", 0.5),
         "p_out": W.integer_array(g, (k_out, n_out), -1, 1, "bf16", 0.5),
         "mask": W.mask_from_lengths(np.array([100, 37, 64]), T)}
    got = _run(d, "f32")
    want = oracle.project_factored(d["x"], d["dy"], d["p_in"], d["p_out"], d["mask"])
    assert np.abs(want).max() < 2 ** 24
    assert np.array_equal(got.astype(np.float64), want)


def test_project_masked_garbage_and_determinism():
    from gpu_util import say
    say("[project] NaN/Inf in masked slots; determinism")
    d = _inputs("asym_bf16_ragged", seed=5)
    a = _run(d, "f32")
    b = _run(d, "f32", poison=True)
    c = _run(d, "f32")
    assert np.all(np.isfinite(b))
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert np.array_equal(a.view(np.uint32), c.view(np.uint32))


def test_project_store_stride_untouched():
    """Rows land at b * g_ld; the store's other columns are left alone."""
    from gpu_util import say
    say("[project] store stride")
    d = _inputs("tiny_f32")
    got = _run(d, "f32", g_ld=100)
    assert np.all(got[:, 64:] == 7.0)
    want = oracle.project_factored(d["x"], d["dy"], d["p_in"], d["p_out"], d["mask"])
    assert np.abs(got[:, :64] - want).max() <= 1e-4 * np.abs(want).max()


def test_project_grouped_equals_single():
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, say
    say("[project] grouped launch == per-layer launches")
    shapes = [(256, 512), (512, 128), (128, 384)]
    B, T, k = 4, 90, 16
    lens = np.array([90, 3, 64, 0])
    mask = dev(W.mask_from_lengths(lens, T))
    layers = []
    store_g = torch.zeros((B, 3 * k * k + 8), dtype=torch.bfloat16, device="cuda")
    store_s = torch.zeros_like(store_g)
    for i, (ni, no) in enumerate(shapes):
        d = W.layer_inputs(9, i, B, T, ni, no, k, k, 1.0, 1.0, "bf16")
        t = {key: dev(d[key]) for key in ("x", "dy", "p_in", "p_out")}
        layers.append(dict(t, g_out=store_g[:, i * k * k:(i + 1) * k * k]))
        P.logra_project_layer(t["x"], t["dy"], t["p_in"], t["p_out"], store_s[:, i * k * k:(i + 1) * k * k],
                              mask=mask)
    P.logra_project_layers(layers, mask=mask)
    torch.cuda.synchronize()
    assert np.array_equal(host(store_g), host(store_s))


def test_project_grouped_multichunk_vs_oracle():
    """A group whose layers span several column chunks per side (chunks of
    14,336 columns), with partial last chunks of different widths (the launch
    processes the chunk slots widest first), against the oracle layer by layer."""
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, rowwise_normwise, say
    say("[project] grouped multi-chunk layers vs oracle")
    shapes = [(30000, 1024), (1024, 20000), (4096, 4096)]
    B, T, k = 2, 70, 16
    lens = np.array([70, 41])
    mask_np = W.mask_from_lengths(lens, T)
    mask = dev(mask_np)
    D = k * k
    store = torch.zeros((B, len(shapes) * D), dtype=torch.float32, device="cuda")
    layers, data = [], []
    for i, (ni, no) in enumerate(shapes):
        d = W.layer_inputs(11, i, B, T, ni, no, k, k, 1.0, 1e-2, "bf16")
        data.append(d)
        t = {key: dev(d[key]) for key in ("x", "dy", "p_in", "p_out")}
        layers.append(dict(t, g_out=store[:, i * D:(i + 1) * D]))
    P.logra_project_layers(layers, mask=mask)
    torch.cuda.synchronize()
    got = host(store).astype(np.float64)
    for i, d in enumerate(data):
        want = oracle.project_factored(d["x"], d["dy"], d["p_in"], d["p_out"], mask_np)
        g = got[:, i * D:(i + 1) * D]
        err = rowwise_normwise(g, want)   # per example: max |diff| / max |oracle|
        say(f"  layer {i} {shapes[i]}: normwise err per example {err:.2e}")
        assert err <= 1e-3


def test_project_scattered_mask_vs_oracle():
    """Masks that are not length prefixes: random holes, a fully masked tile
    between valid ones, tiles whose only valid token is the first or the last
    of the tile, and a ragged last tile holding one valid token.  NaN and -Inf
    in every masked slot must not reach the result, and a layer spans two
    chunks on the x side.  Grouped launch, fp32 out, against the oracle."""
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, say
    say("[project] scattered masks with poisoned masked slots vs oracle")
    B, T = 3, 300                                     # five tiles, the last one 44 tokens
    mask_np = (W.rng(3, 41, 0).random((B, T)) < 0.6).astype(np.uint8)
    mask_np[0, 64:128] = 0                            # fully masked tile between valid ones
    mask_np[1, :] = 0
    mask_np[1, 64] = 1                                # first token of tile 1 only
    mask_np[1, 255] = 1                               # last token of tile 3 only
    mask_np[2, 256:] = 0
    mask_np[2, 299] = 1                               # last token of the ragged tile only
    shapes = [(6400, 96), (200, 328)]
    k_in, k_out = 12, 20
    D = k_in * k_out
    store = torch.zeros((B, len(shapes) * D), dtype=torch.float32, device="cuda")
    layers, data = [], []
    bad = mask_np == 0
    for i, (ni, no) in enumerate(shapes):
        d = W.layer_inputs(13, i, B, T, ni, no, k_in, k_out, 1.0, 0.5, "bf16")
        data.append(d)
        x, dy = d["x"].copy(), d["dy"].copy()
        x[bad] = 0x7FC0                               # NaN
        dy[bad] = 0xFF80                              # -Inf
        layers.append(dict(x=dev(x), dy=dev(dy), p_in=dev(d["p_in"]), p_out=dev(d["p_out"]),
                           g_out=store[:, i * D:(i + 1) * D]))
    P.logra_project_layers(layers, mask=dev(mask_np))
    torch.cuda.synchronize()
    got = host(store).astype(np.float64)
    assert np.all(np.isfinite(got))
    for i, d in enumerate(data):
        want = oracle.project_factored(d["x"], d["dy"], d["p_in"], d["p_out"], mask_np)
        g = got[:, i * D:(i + 1) * D]
        for b in range(B):
            err = np.linalg.norm(g[b] - want[b]) / np.linalg.norm(want[b])
            say(f"  layer {i} {shapes[i]} example {b} ({int(mask_np[b].sum())} tokens): normwise err {err:.2e}")
            assert err <= 1e-3


@pytest.mark.parametrize("k,shared", [(16, False), (16, True), (64, False)])
def test_project_largest_group_equals_single(k, shared):
    """A grouped launch of the most layers it takes (48: the packed per-layer
    table, layer indices past 15 in the slot order), with layers of many
    widths, some of them multi-chunk at k = 16, a ragged mask, and at k = 16
    groups of layers given the same x (shared passes): every output equals
    bit for bit the output of the same layer projected in a launch of its
    own, and sampled layers match the oracle."""
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, normwise, say
    nl = P.MAX_GROUP
    g = W.rng(81, k, int(shared))
    B, T = 3, 130
    widths = [64, 200, 768, 1000, 6144 + 128, 96]
    shapes = [(widths[(i // 2) % 6], widths[(i * 5 + 2) % 6]) for i in range(nl)]   # pairs share a width
    if k == 64:   # the wide layers only in the first half, to keep the test small
        shapes = [(ni if i < 24 else min(ni, 1000), no if i < 24 else min(no, 1000)) for i, (ni, no) in enumerate(shapes)]
    say(f"[project] {nl} layers in one launch at k={k}, shared inputs {shared}, B={B} T={T}")
    lens = W.lengths(g, B, 1, T)
    mask_np = W.mask_from_lengths(lens, T)
    mask = dev(mask_np)
    xs, ins = [], []
    for i, (ni, no) in enumerate(shapes):
        if shared and i % 2 == 1:   # the same tensor as the layer before: one shared pass
            xs.append(xs[-1])
            ins.append(ins[-1])
        else:
            xs.append(W.normal(g, (B, T, ni), 1.0, "bf16"))
            ins.append(dev(xs[-1]))
    dys = [W.normal(g, (B, T, no), 1e-2, "bf16") for _, no in shapes]
    pis = [W.projection(g, k, ni, "bf16") for ni, _ in shapes]
    pos = [W.projection(g, k, no, "bf16") for _, no in shapes]
    D = k * k
    store_g = torch.full((B, nl * D), np.nan, dtype=torch.float32, device="cuda")
    store_s = torch.full_like(store_g, np.nan)
    layers = []
    for i in range(nl):
        t = dict(x=ins[i], dy=dev(dys[i]), p_in=dev(pis[i]), p_out=dev(pos[i]))
        layers.append(dict(t, g_out=store_g[:, i * D:(i + 1) * D]))
        P.logra_project_layer(t["x"], t["dy"], t["p_in"], t["p_out"], store_s[:, i * D:(i + 1) * D], mask=mask)
    P.logra_project_layers(layers, mask=mask)
    torch.cuda.synchronize()
    got_g, got_s = host(store_g), host(store_s)
    assert np.array_equal(got_g.view(np.uint32), got_s.view(np.uint32))
    for i in (0, 17, nl - 1):
        want = oracle.project_factored(xs[i], dys[i], pis[i], pos[i], mask_np)
        err = max(normwise(got_g[b, i * D:(i + 1) * D], want[b]) for b in range(B))
        say(f"  layer {i} ({shapes[i][0]}->{shapes[i][1]}): max normwise err {err:.2e}")
        assert err <= 1e-3


def test_project_shared_inputs_bitwise_equal():
    """Layers given the same x tensor (q/k/v and gate/up of a transformer
    block) are projected from one pass over x; every output must equal, bit
    for bit, the output of the same layers given separate copies of x (each
    projection sees the same operands in the same order), and the oracle."""
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, normwise, say
    say("[project] shared inputs: one pass over x for q/k/v and for gate/up")
    g = W.rng(80)
    B, T, k = 3, 150, 16
    shapes = [("q", 512, 512), ("k", 512, 128), ("v", 512, 128), ("o", 512, 512), ("gate", 512, 1024),
              ("up", 512, 1024), ("down", 1024, 512)]
    lens = W.lengths(g, B, 1, T)
    mask_np = W.mask_from_lengths(lens, T)
    mask = dev(mask_np)
    x_attn = W.normal(g, (B, T, 512), 1.0, "bf16")
    x_mlp = W.normal(g, (B, T, 512), 1.0, "bf16")
    x_o = W.normal(g, (B, T, 512), 1.0, "bf16")
    x_down = W.normal(g, (B, T, 1024), 1.0, "bf16")
    xs = [x_attn, x_attn, x_attn, x_o, x_mlp, x_mlp, x_down]
    dys = [W.normal(g, (B, T, no), 1e-2, "bf16") for _, _, no in shapes]
    pis = [W.projection(g, k, ni, "bf16") for _, ni, _ in shapes]
    pos = [W.projection(g, k, no, "bf16") for _, _, no in shapes]
    xa, xm = dev(x_attn), dev(x_mlp)
    shared_x = [xa, xa, xa, dev(x_o), xm, xm, dev(x_down)]          # the same tensors: shared
    copies_x = [dev(x) for x in xs]                                  # separate copies: not shared
    outs = []
    for xlist in (shared_x, copies_x):
        store = torch.full((B, 7 * k * k), np.nan, dtype=torch.float32, device="cuda")
        layers = [dict(x=xlist[j], dy=dev(dys[j]), p_in=dev(pis[j]), p_out=dev(pos[j]),
                       g_out=store[:, j * k * k:(j + 1) * k * k]) for j in range(7)]
        P.logra_project_layers(layers, mask=mask)
        torch.cuda.synchronize()
        outs.append(host(store))
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
    for j in (0, 2, 5):
        want = oracle.project_factored(xs[j], dys[j], pis[j], pos[j], mask_np)
        err = max(normwise(outs[0][b, j * k * k:(j + 1) * k * k], want[b]) for b in range(B))
        say(f"  {shapes[j][0]}: max normwise err {err:.2e}")
        assert err <= 1e-3


@pytest.mark.parametrize("k", [16, 32, 64])
def test_project_paired_equals_unpaired(k):
    """With every layer side in one chunk, a workgroup runs a tile's (k <= 16,
    stream kernel) or a tile group's (16 < k <= 64, tile-group kernel) x and dy
    items back to back and forms the tile sums itself (the tile-sum kernel is
    skipped; the example sums skip empty tiles).  A layer wider than one chunk
    turns that off for the whole launch.  The narrow layers' outputs must be
    the same bits either way, and match the oracle."""
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, normwise, say
    say(f"[project] paired items == unpaired (one wide layer in the launch), k={k}")
    g = W.rng(83)
    B, T = 5, 200
    narrow = [(768, 2304), (768, 768), (3072, 768)]
    wide = (512, 16384)           # two chunks on its dy side (chunks of 14,336 columns)
    lens = W.lengths(g, B, 1, T)
    lens[1], lens[-1] = 0, T      # an empty example and a full one
    mask_np = W.mask_from_lengths(lens, T)
    mask = dev(mask_np)
    data = [W.layer_inputs(84, i, B, T, ni, no, k, k, 1.0, 1e-2, "bf16") for i, (ni, no) in enumerate(narrow + [wide])]
    t = [{key: dev(d[key]) for key in ("x", "dy", "p_in", "p_out")} for d in data]
    outs = []
    for with_wide in (False, True):
        n = len(narrow) + int(with_wide)
        store = torch.full((B, n * k * k), np.nan, dtype=torch.float32, device="cuda")
        layers = [dict(t[i], g_out=store[:, i * k * k:(i + 1) * k * k]) for i in range(n)]
        P.logra_project_layers(layers, mask=mask)
        torch.cuda.synchronize()
        outs.append(host(store)[:, :len(narrow) * k * k])
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
    assert np.all(outs[0][1] == 0.0)          # the empty example
    for i in (0, 2):
        d = data[i]
        want = oracle.project_factored(d["x"], d["dy"], d["p_in"], d["p_out"], mask_np)
        err = max(normwise(outs[0][b, i * k * k:(i + 1) * k * k], want[b]) for b in range(B) if lens[b] > 0)
        say(f"  layer {narrow[i]}: equal bits paired and unpaired; max normwise err {err:.2e}")
        assert err <= 1e-3


@pytest.mark.parametrize("k", [16, 64])
def test_project_all_masked_batch_writes_zeros(k):
    """No valid token anywhere: no tile is listed and no item runs (k = 16: the
    paired stream kernel; k = 64: the paired tile-group kernel); every output
    row (pre-filled with 7.0) must still be written as zeros."""
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, say
    say(f"[project] fully masked batch, k={k}")
    B, T = 3, 130
    d = W.layer_inputs(12, 0, B, T, 256, 320, k, k, 1.0, 1.0, "bf16", np.zeros(B, dtype=np.int64))
    for out in (torch.float32, torch.bfloat16):
        store = torch.full((B, k * k + 5), 7.0, dtype=out, device="cuda")
        P.logra_project_layer(dev(d["x"]), dev(d["dy"]), dev(d["p_in"]), dev(d["p_out"]), store[:, :k * k],
                              mask=dev(d["mask"]))
        torch.cuda.synchronize()
        got = host(store).astype(np.float64) if out == torch.float32 else W.bf16_bits_to_f32(host(store))
        assert np.all(got[:, :k * k] == 0.0) and np.all(got[:, k * k:] == 7.0)


def test_project_many_examples_vs_oracle():
    """B = 1100 short examples (1100 tiles: the tile listing and the per-example
    bookkeeping take more than one pass of the 1024-thread prep workgroup),
    a fifth of them fully masked, k = 24 (two 16-wide projection blocks)."""
    from gpu_util import rowwise_normwise, say
    say("[project] B = 1100 examples, ragged, some fully masked")
    B, T = 1100, 40
    g = W.rng(13)
    lens = W.lengths(g, B, 0, T)
    lens[g.random(B) < 0.2] = 0
    d = W.layer_inputs(13, 1, B, T, 96, 160, 24, 20, 1.0, 1.0, "bf16", lens)
    got = _run(d, "f32")
    want = oracle.project_factored(d["x"], d["dy"], d["p_in"], d["p_out"], d["mask"])
    err = rowwise_normwise(got, want)
    say(f"  normwise err {err:.2e}")
    assert err <= 1e-3
    assert np.all(got[lens == 0] == 0.0)


def test_project_reused_workspace_across_masks():
    """One workspace, filled with garbage first, serves consecutive grouped
    launches with different masks: the launch clears its own counters, and
    each result equals the oracle's and a fresh-workspace launch bit for bit."""
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, rowwise_normwise, say
    say("[project] workspace reused across launches with different masks")
    B, T, k = 4, 200, 16
    shapes = [(512, 256), (256, 4608)]
    g = W.rng(14)
    data = [W.layer_inputs(14, i, B, T, ni, no, k, k, 1.0, 1e-2, "bf16") for i, (ni, no) in enumerate(shapes)]
    tens = [{key: dev(d[key]) for key in ("x", "dy", "p_in", "p_out")} for d in data]
    D = k * k
    descs = (P.LayerDesc * 2)(*[P.LayerDesc(0, 0, 0, 0, 0, ni, no) for ni, no in shapes])
    ws = torch.full((P.logra_project_layers_ws_size(descs, 2, B, T, k, k),), 0x7F, dtype=torch.uint8, device="cuda")
    for trial in range(3):
        lens = W.lengths(g, B, 0, T)
        lens[trial % B] = 0
        mask_np = W.mask_from_lengths(lens, T)
        outs = []
        for w in (ws, None):
            store = torch.full((B, 2 * D), np.nan, dtype=torch.float32, device="cuda")
            layers = [dict(t, g_out=store[:, i * D:(i + 1) * D]) for i, t in enumerate(tens)]
            P.logra_project_layers(layers, mask=dev(mask_np), ws=w)
            torch.cuda.synchronize()
            outs.append(host(store))
        assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32)), trial
        for i, d in enumerate(data):
            want = oracle.project_factored(d["x"], d["dy"], d["p_in"], d["p_out"], mask_np)
            gi = outs[0][:, i * D:(i + 1) * D].astype(np.float64)
            assert rowwise_normwise(gi[lens > 0], want[lens > 0]) <= 1e-3, (trial, i)
            assert np.all(gi[lens == 0] == 0.0)


def test_project_rejects_out_of_range_row_stride():
    """A row stride that puts the last output row beyond device memory is
    refused on the host (no kernel is launched)."""
    import ctypes
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import say
    say("[project] out-of-range g_ld is rejected")
    B, T, n, k = 2, 64, 64, 4
    x = torch.zeros((B, T, n), dtype=torch.bfloat16, device="cuda")
    pi = torch.zeros((k, n), dtype=torch.bfloat16, device="cuda")
    g = torch.zeros((B, k * k), dtype=torch.float32, device="cuda")
    ws = torch.empty(P.logra_project_ws_size(B, T, n, n, k, k), dtype=torch.uint8, device="cuda")
    L = P.lib()

    def call(g_ld):
        return L.logra_project_layer(ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(x.data_ptr()), P.BF16, B, T, n,
                                     n, None, ctypes.c_void_p(pi.data_ptr()), ctypes.c_void_p(pi.data_ptr()), k, k,
                                     ctypes.c_void_p(g.data_ptr()), P.F32, g_ld, ctypes.c_void_p(ws.data_ptr()),
                                     ws.numel(), None)
    assert call(1 << 47) == P.ERR_INVALID_ARG and "exceed device memory" in P.logra_last_error()
    assert call(1 << 40) == P.ERR_INVALID_ARG and "last row of g_out" in P.logra_last_error()
