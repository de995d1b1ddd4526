"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Bar: selected and admitted index sets bit-exact, theta equal in fp64, index
digests and certificate scalars bit-exact, attention outputs within 2e-2
relative L2 per (b, h) and lse within 1e-3.  Sizes span several tiles and a
ragged tail; the full-size configs are checked on sampled sequences.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_03949_amd as vkv
from paper_2609_03949_amd import synth

import _checks
from _harness import gpu_index, gpu_step, host_inputs, index_cols, oracle_step, rel_l2

pytestmark = pytest.mark.gpu

OUT_TOL = _checks.OUT_TOL
LSE_TOL = _checks.LSE_TOL


def say(msg):
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def ctx():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    vkv.load()
    c = vkv.Context(0)
    yield c
    c.close()


def check_step(wl, g, o, seqs, two_tier=False):
    return _checks.check_step(g, o, seqs, two_tier)


# ------------------------------------------------------------ index build

@pytest.mark.parametrize("basis,r,with_rope", [
    ("orthonormal", 64, True), ("gaussian", 64, True), ("orthonormal", 256, False),
    ("identity", 512, True), ("zero", 64, True), ("orthonormal", 32, False),
])
def test_digest_build_bit_exact(ctx, basis, r, with_rope):
    say(f"digest_build basis={basis} r={r} rope={with_rope}")
    cfg = synth.CONFIGS["cfg3"].with_(H=4)
    wl = synth.make_workload(cfg, "cuda", B=2, T=1000)
    P = synth.make_basis(basis, r).cuda()
    cert = basis != "gaussian"          # the Gaussian basis is not contractive
    cache = wl["cache"]
    cols = (64 if with_rope else 0) + r
    index = torch.empty(2, 1000, cols, dtype=torch.bfloat16, device="cuda")
    eta = torch.empty(2, 1000, device="cuda") if cert else None
    eps = torch.empty(2, 1000, device="cuda") if cert else None
    gam = torch.empty(2, 1000, device="cuda") if cert else None
    vkv.digest_build(ctx, cache, P, r, with_rope, index, eta, eps, gam)
    torch.cuda.synchronize()
    ci = synth.to_numpy_bits(cache)
    Pi = synth.to_numpy_bits(P)
    oi, oe, oep, og = oracle.digest_build(ci, Pi, r, with_rope=with_rope, scalars=cert)
    assert np.array_equal(synth.to_numpy_bits(index), oi)
    if cert:
        assert np.array_equal(eta.cpu().numpy().view(np.uint32), oe.view(np.uint32))
        assert np.array_equal(eps.cpu().numpy().view(np.uint32), oep.view(np.uint32))
        assert np.array_equal(gam.cpu().numpy().view(np.uint32), og.view(np.uint32))


@pytest.mark.parametrize("r,cert", [(160, True), (64, False)])
def test_digest_build_bit_exact_under_rounding(ctx, r, cert):
    """Index digests and row scalars against the oracle, bit for bit, with latent
    rows spread over 2^60 and a small-entry basis (contractive, so the
    certificate mode runs): the fp64 sums round at many steps, so only the
    i-ascending order reproduces them."""
    say(f"digest_build rounding r={r} cert={cert}")
    rng = np.random.default_rng(5 + r)
    B, T = 2, 700
    cache = _wide_bf16(rng, (B, T, 576), -30, 30).cuda()
    P = _wide_bf16(rng, (r, 512), -24, -14).cuda()
    index = torch.empty(B, T, 64 + r, dtype=torch.bfloat16, device="cuda")
    eta = torch.empty(B, T, device="cuda") if cert else None
    eps = torch.empty(B, T, device="cuda") if cert else None
    gam = torch.empty(B, T, device="cuda") if cert else None
    vkv.digest_build(ctx, cache, P, r, True, index, eta, eps, gam)
    torch.cuda.synchronize()
    ci = synth.to_numpy_bits(cache)
    Pi = synth.to_numpy_bits(P)
    oi, oe, oep, og = oracle.digest_build(ci, Pi, r, with_rope=True, scalars=cert)
    assert np.array_equal(synth.to_numpy_bits(index), oi)
    if cert:
        assert np.array_equal(eta.cpu().numpy().view(np.uint32), oe.view(np.uint32))
        assert np.array_equal(eps.cpu().numpy().view(np.uint32), oep.view(np.uint32))
        assert np.array_equal(gam.cpu().numpy().view(np.uint32), og.view(np.uint32))
    # the inputs separate summation orders (sequential vs blocked fp64 sums)
    c = cache[0, :64, :512].cpu().float().numpy().astype(np.float64)
    Pf = P.cpu().float().numpy().astype(np.float64)
    y_seq = np.zeros((64, r))
    for i in range(512):
        y_seq = y_seq + c[:, i:i + 1] * Pf[None, :, i]
    y_blk = np.zeros((64, r))
    for i0 in range(0, 512, 64):
        y_blk = y_blk + c[:, i0:i0 + 64] @ Pf[:, i0:i0 + 64].T
    assert np.count_nonzero(y_seq != y_blk) > 0


def test_digest_build_refuses_non_contractive_basis(ctx):
    say("digest_build non-contractive")
    wl = synth.make_workload(synth.CONFIGS["cfg0"].with_(H=2), "cuda", T=256)
    P = synth.make_basis("gaussian", 64).cuda()     # ||P||_2 ~ 3.8
    index = torch.full((1, 256, 128), 7, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    eta = torch.full((1, 256), 5.0, device="cuda")
    eps = torch.full_like(eta, 5.0)
    gam = torch.full_like(eta, 5.0)
    with pytest.raises(vkv.VkvError) as ei:
        vkv.digest_build(ctx, wl["cache"], P, 64, True, index, eta, eps, gam)
    assert ei.value.code == -5
    torch.cuda.synchronize()
    assert torch.all(eta == 5.0) and torch.all(index.view(torch.int16) == 7)


# ------------------------------------------------------------ query prep

def _wide_bf16(rng, shape, lo, hi):
    """bf16-representable values sign * (1 + m/128) * 2^e, e uniform in [lo, hi):
    the fp64 sums of their products round at many steps, so a summation
    order other than i ascending changes some results."""
    m = rng.integers(0, 128, shape)
    e = rng.integers(lo, hi, shape)
    sg = rng.choice([-1.0, 1.0], shape)
    return torch.from_numpy((sg * np.ldexp(1.0 + m / 128.0, e)).astype(np.float32)).to(torch.bfloat16)


@pytest.mark.parametrize("mode,r", [(synth.MODE_ROPE_DIGEST, 64), (synth.MODE_ROPE_DIGEST, 160),
                                    (synth.MODE_DIGEST, 512), (synth.MODE_ROPE, 0)])
def test_query_prep_bit_exact_under_rounding(ctx, mode, r):
    """qt and the head certificate scalars against the oracle, bit for bit, with
    queries and basis spread over 2^60: the projection and ||q||^2 are fp64
    chains with i ascending (white-box: qt and the scalars are read from the
    first two regions of the workspace)."""
    say(f"query prep rounding mode={mode} r={r}")
    rng = np.random.default_rng(11 + r)
    B, H, T = 2, 24, 64
    q_lat = _wide_bf16(rng, (B, H, 512), -30, 30)
    q_rope = _wide_bf16(rng, (B, H, 64), -8, 8)
    P = _wide_bf16(rng, (max(r, 1), 512), -20, 20) if r else None
    cache = torch.from_numpy(rng.standard_normal((B, T, 576)).astype(np.float32)).to(torch.bfloat16)
    dev = "cuda"
    q_lat, q_rope, cache = q_lat.to(dev), q_rope.to(dev), cache.to(dev)
    Pd = P.to(dev) if P is not None else None
    cols, has_rope = index_cols(mode, r)
    index = torch.zeros(B, T, cols, dtype=torch.bfloat16, device=dev) if cols else None
    step = vkv.Step(cache, q_lat, q_rope, 0, mode, r, index=index, index_has_rope=has_rope, P=Pd)
    ws = vkv.alloc_workspace(step, 1)
    vkv.query_prep(ctx, step, ws)
    torch.cuda.synchronize()
    n = (64 if mode & 1 else 0) + (r if mode & 2 else 0)
    nb = B * H * n * 2
    qt = ws[:nb].cpu().numpy().view(np.uint16).reshape(B, H, n)
    h0 = (nb + 255) // 256 * 256
    hsc = ws[h0:h0 + B * H * 16].cpu().numpy().view(np.float32).reshape(B, H, 4)
    Pb = synth.to_numpy_bits(P) if P is not None else None
    qt_o, a_o, n_o, e_o = oracle.query_prep(synth.to_numpy_bits(q_lat.cpu()), synth.to_numpy_bits(q_rope.cpu()),
                                            Pb, r, mode)
    assert np.array_equal(qt, qt_o)
    assert np.array_equal(hsc[..., 0], a_o)
    assert np.array_equal(hsc[..., 1], n_o)
    assert np.array_equal(hsc[..., 2], e_o)
    if r:
        # the inputs do separate summation orders: the sequential fp64 sums
        # (products exact, one rounding per term) differ from a blocked order
        ql = q_lat.cpu().float().numpy().astype(np.float64)
        Pf = P.float().numpy().astype(np.float64)
        w_seq = np.zeros((B, H, r))
        for i in range(512):
            w_seq = w_seq + ql[:, :, i:i + 1] * Pf[None, None, :, i]
        w_blk = np.zeros((B, H, r))
        for i0 in range(0, 512, 64):
            w_blk = w_blk + np.einsum("bhi,ji->bhj", ql[:, :, i0:i0 + 64], Pf[:, i0:i0 + 64])
        assert np.count_nonzero(w_seq != w_blk) > 0


# ------------------------------------------------------ reduced configs

REDUCED = [
    ("cfg0", dict(T=5000)),
    ("cfg1", dict(B=3, T=6000)),
    ("cfg2_r64", dict(B=2, T=7000)),
    ("cfg2_r192", dict(B=2, T=7000)),
    ("cfg2_r256", dict(B=2, T=7000)),
    ("cfg4", dict(B=3, T=9000)),
]


@pytest.mark.parametrize("name,kw", REDUCED)
def test_step_parity_reduced(ctx, name, kw):
    cfg = synth.CONFIGS[name]
    say(f"step parity {name} {kw}")
    wl = synth.make_workload(cfg, "cuda", **kw)
    k = max(1, wl["A"] // 32) if name != "cfg0" else wl["A"] // 8
    g, _ = gpu_step(ctx, wl, k=k)
    seqs = list(range(wl["B"]))
    o, _ = oracle_step(wl, seqs, k=k)
    check_step(wl, g, o, seqs)


def test_step_parity_two_tier_reduced(ctx):
    cfg = synth.CONFIGS["cfg3"]
    say("two-tier parity cfg3 reduced")
    wl = synth.make_workload(cfg, "cuda", B=2, T=5000)
    k = wl["A"] // 32
    g, _ = gpu_step(ctx, wl, k=k, two_tier=True)
    o, _ = oracle_step(wl, [0, 1], k=k, two_tier=True)
    check_step(wl, g, o, [0, 1], two_tier=True)


@pytest.mark.parametrize("basis,r,H", [("identity", 448, 16), ("orthonormal", 256, 8),
                                       ("identity", 512, 4)])
def test_two_tier_partial_admission(ctx, basis, r, H):
    """A basis that captures most of the latent makes the bound tight enough
    that only some rows are admitted: exercises the fp64 band decisions."""
    say(f"two-tier partial basis={basis} r={r} H={H}")
    cfg = synth.CONFIGS["cfg3"].with_(H=H, r=r, rows="gaussian", needles=4)
    wl = synth.make_workload(cfg, "cuda", B=2, T=3000, basis=basis)
    k = 60
    g, _ = gpu_step(ctx, wl, k=k, two_tier=True)
    o, _ = oracle_step(wl, [0, 1], k=k, two_tier=True)
    check_step(wl, g, o, [0, 1], two_tier=True)


def test_admitted_splits_taken_in_turn(ctx):
    """Many sequences and a near-total admission: the admitted rows' splits
    outnumber the workgroups kept for them, so some workgroups take two
    splits in turn (64 sequences of 16 heads leave 4 workgroups per sequence;
    a capacity of 19744 rows makes 20 admitted splits of 1024 rows, taken by
    16 workgroups).  Sampled sequences against the oracle."""
    say("admitted splits taken in turn by a bounded set of workgroups")
    cfg = synth.CONFIGS["cfg3"].with_(H=16)
    wl = synth.make_workload(cfg, "cuda", B=64, T=20000)
    k = 256
    g, _ = gpu_step(ctx, wl, k=k, two_tier=True)
    seqs = [0, 21, 63]
    adm = g["adm_count"]
    say(f"  admitted rows per sequence: min {int(adm.min())} max {int(adm.max())} of {wl['A'] - k}")
    # the base splits cover 576 positions (3 x 192), so more than 16 admitted
    # splits of 1024 rows hold rows once k + W + admitted - 576 > 16 x 1024
    assert int(adm.min()) + k + wl["W"] - 576 > 16 * 1024
    o, _ = oracle_step(wl, seqs, k=k, two_tier=True)
    check_step(wl, g, o, seqs, two_tier=True)


def test_two_tier_capacity_overflow(ctx):
    say("two-tier capacity overflow")
    cfg = synth.CONFIGS["cfg3"].with_(H=8)
    wl = synth.make_workload(cfg, "cuda", B=2, T=2000)
    k = 50
    cap = 100
    g, _ = gpu_step(ctx, wl, k=k, two_tier=True, cap=cap)
    o, _ = oracle_step(wl, [0, 1], k=k, two_tier=True, cap=cap)
    for b in (0, 1):
        assert g["adm_count"][b] == o[b]["adm_count"] > cap
        assert np.array_equal(g["adm"][b, :cap], o[b]["adm"][:cap])
    check_step(wl, g, o, [0, 1], two_tier=True)


# ------------------------------------------------------------ edge cases

@pytest.mark.parametrize("H", [1, 8, 24, 64, 128])
def test_head_counts(ctx, H):
    say(f"heads H={H}")
    cfg = synth.CONFIGS["cfg4"].with_(H=H)
    wl = synth.make_workload(cfg, "cuda", B=2, T=3000)
    g, _ = gpu_step(ctx, wl, k=97)
    o, _ = oracle_step(wl, [0, 1], k=97)
    check_step(wl, g, o, [0, 1])


@pytest.mark.parametrize("mode,r", [(synth.MODE_DIGEST, 32), (synth.MODE_DIGEST, 512),
                                    (synth.MODE_ROPE_DIGEST, 128), (synth.MODE_ROPE_DIGEST, 512),
                                    (synth.MODE_ROPE_DIGEST, 256)])
def test_widths(ctx, mode, r):
    say(f"width mode={mode} r={r}")
    cfg = synth.CONFIGS["cfg2_r64"].with_(mode=mode, r=r, H=16)
    wl = synth.make_workload(cfg, "cuda", B=2, T=2500)
    g, _ = gpu_step(ctx, wl, k=77)
    o, _ = oracle_step(wl, [0, 1], k=77)
    check_step(wl, g, o, [0, 1])


@pytest.mark.parametrize("k", [0, 1, 2, "A-1", "A"])
def test_budget_extremes(ctx, k):
    say(f"budget k={k}")
    cfg = synth.CONFIGS["cfg0"].with_(H=16)
    wl = synth.make_workload(cfg, "cuda", T=2100)
    kk = {"A-1": wl["A"] - 1, "A": wl["A"]}.get(k, k)
    g, _ = gpu_step(ctx, wl, k=kk)
    o, _ = oracle_step(wl, [0], k=kk)
    check_step(wl, g, o, [0])


def test_full_budget_is_dense_attention(ctx):
    """k = A attends every row: the output is dense attention (kill-switch)."""
    say("k = A dense")
    cfg = synth.CONFIGS["cfg4"].with_(H=32)
    wl = synth.make_workload(cfg, "cuda", B=1, T=3000)
    g, _ = gpu_step(ctx, wl, k=wl["A"])
    cache, q_lat, q_rope, _ = host_inputs(wl, [0])
    out, lse = oracle.attend(q_lat[0], q_rope[0], cache[0], np.arange(wl["T"], dtype=np.int32),
                             wl["scale"])
    assert rel_l2(g["out"][0], out) < OUT_TOL
    assert np.max(np.abs(g["lse"][0] - lse)) < LSE_TOL


def test_single_attended_row_is_bit_exact(ctx):
    say("single row")
    cfg = synth.CONFIGS["cfg0"].with_(H=16, W=0)
    wl = synth.make_workload(cfg, "cuda", T=700)
    g, _ = gpu_step(ctx, wl, k=1)
    o, _ = oracle_step(wl, [0], k=1)
    u = int(o[0]["sel"][0])
    assert g["sel"][0][0] == u
    cache, _, _, _ = host_inputs(wl, [0])
    want = np.repeat(cache[0, u:u + 1, :512], 16, axis=0)
    assert np.array_equal(g["out_bits"][0], want)


def test_empty_attended_set(ctx):
    say("empty set")
    cfg = synth.CONFIGS["cfg0"].with_(H=4, W=0)
    wl = synth.make_workload(cfg, "cuda", T=300)
    g, _ = gpu_step(ctx, wl, k=0)
    assert np.all(g["out"][0] == 0) and np.all(np.isneginf(g["lse"][0]))


def test_no_archive(ctx):
    say("W = T")
    cfg = synth.CONFIGS["cfg4"].with_(H=16, W=512)
    wl = synth.make_workload(cfg, "cuda", B=2, T=512)
    g, _ = gpu_step(ctx, wl, k=0)
    o, _ = oracle_step(wl, [0, 1], k=0)
    check_step(wl, g, o, [0, 1])


def test_all_equal_keys_take_lowest_indices(ctx):
    """q_rope = 0 and a zero digest query: every key ties at 0."""
    say("all ties")
    cfg = synth.CONFIGS["cfg1"].with_(H=8)
    wl = synth.make_workload(cfg, "cuda", B=2, T=3000)
    wl["q_rope"].zero_()
    g, _ = gpu_step(ctx, wl, k=300)
    for b in range(2):
        assert np.array_equal(g["sel"][b], np.arange(300))
        assert g["theta"][b] == 0.0
    o, _ = oracle_step(wl, [0, 1], k=300)
    check_step(wl, g, o, [0, 1])


def test_duplicated_rows_and_near_ties(ctx):
    """Rows duplicated many times (exact ties of the exact key) and rows a
    few ulps apart at the threshold."""
    say("duplicates / near ties")
    cfg = synth.CONFIGS["cfg4"].with_(H=16)
    wl = synth.make_workload(cfg, "cuda", B=2, T=4000)
    c = wl["cache"]
    src = torch.randint(0, 50, (3000,), generator=torch.Generator().manual_seed(3)).cuda()
    c[:, :3000] = c[:, src]
    # perturb some copies by one bf16 ulp in one coordinate
    bits = c.view(torch.int16)
    bits[:, 1000:1200, 5] += 1
    g, _ = gpu_step(ctx, wl, k=400)
    o, _ = oracle_step(wl, [0, 1], k=400)
    check_step(wl, g, o, [0, 1])


def test_bracket_missed_by_the_sample(ctx):
    """The largest keys sit only at rows the strided key sample never reads
    (A = 16384: the sample takes every 4th row); the counting pass finds the
    sampled bracket wrong and redoes the histogram over the whole key range."""
    say("sample miss")
    cfg = synth.CONFIGS["cfg1"].with_(H=16, needles=0)
    wl = synth.make_workload(cfg, "cuda", B=1, T=16384 + 256)
    rows = torch.arange(1, 4096, 4, device="cuda")
    wl["cache"][0, rows, 512:] = (wl["cache"][0, rows, 512:].float() * 8).to(torch.bfloat16)
    g, _ = gpu_step(ctx, wl, k=256)
    o, _ = oracle_step(wl, [0], k=256)
    check_step(wl, g, o, [0])
    assert set(g["sel"][0].tolist()) <= set(rows.tolist())


def test_bracket_missed_by_the_sample_long_archive(ctx):
    """The same miss on an archive of 65536 rows: the sample takes runs of 32
    rows about 1040 apart, so rows 40..940 are never sampled; the largest keys
    are planted there, and the bracket pass must fall back to the whole key
    range of 32 counting blocks' worth of keys."""
    say("sample miss, long archive")
    cfg = synth.CONFIGS["cfg1"].with_(H=16, needles=0)
    wl = synth.make_workload(cfg, "cuda", B=1, T=65536 + 256)
    rows = torch.arange(40, 940, 3, device="cuda")
    wl["cache"][0, rows, 512:] = (wl["cache"][0, rows, 512:].float() * 8).to(torch.bfloat16)
    g, _ = gpu_step(ctx, wl, k=256)
    o, _ = oracle_step(wl, [0], k=256)
    check_step(wl, g, o, [0])
    assert set(g["sel"][0].tolist()) <= set(rows.tolist())


@pytest.mark.parametrize("H", [16, 128])
def test_identical_heads_make_every_head_a_candidate(ctx, H):
    """All heads carry the same query: every head ties for the maximum of every
    ambiguous row, so all of them go through the fp64 pass (H = 16: as queued
    (row, head) pairs; H = 128: in the re-screening wave itself)."""
    say(f"identical heads H={H}")
    cfg = synth.CONFIGS["cfg4"].with_(H=H)
    wl = synth.make_workload(cfg, "cuda", B=1, T=6000)
    wl["q_lat"][0] = wl["q_lat"][0, :1].expand(H, -1)
    wl["q_rope"][0] = wl["q_rope"][0, :1].expand(H, -1)
    g, _ = gpu_step(ctx, wl, k=500)
    o, _ = oracle_step(wl, [0], k=500)
    check_step(wl, g, o, [0])


def test_cancellation_heavy_scores_stay_within_bound(ctx):
    """Index rows built so that each score is a sum of large terms that cancel:
    the fp32 MFMA key must stay within the certified bound, and selection
    stays exact."""
    say("cancellation")
    cfg = synth.CONFIGS["cfg1"].with_(H=16)
    wl = synth.make_workload(cfg, "cuda", B=1, T=4096)
    r = wl["cache"][0, :, 512:].float()
    big = torch.randn(4096, 32, device="cuda", generator=torch.Generator("cuda").manual_seed(5)) * 64
    r[:, :32] = big
    r[:, 32:] = -big + 1e-2 * torch.randn(4096, 32, device="cuda")
    wl["cache"][0, :, 512:] = r.to(torch.bfloat16)
    q = torch.ones(16, 64, device="cuda") + 1e-3 * torch.randn(16, 64, device="cuda")
    wl["q_rope"][0] = q.to(torch.bfloat16)
    g, _ = gpu_step(ctx, wl, k=128)
    o, _ = oracle_step(wl, [0], k=128)
    key = o[0]["key"]
    cache, _, q_rope, _ = host_inputs(wl, [0])
    xn = np.linalg.norm(oracle.decode_bf16(cache[0, :, 512:]), axis=1).max()
    qn = np.linalg.norm(oracle.decode_bf16(q_rope[0]), axis=1).max()
    bound = 8 * 64 * 2.0 ** -23 * qn * xn
    err = np.max(np.abs(g["key"][0, :wl["A"]].astype(np.float64) - key))
    say(f"max key error {err:.3e}, bound {bound:.3e}")
    assert err <= bound / 8
    check_step(wl, g, o, [0])


@pytest.mark.parametrize("mode,r,H,B,T", [
    (synth.MODE_ROPE_DIGEST, 64, 128, 2, 9000),     # 128 dims, the scan's main shape
    (synth.MODE_ROPE, 0, 128, 2, 7001),             # 64 dims, ragged archive
    (synth.MODE_ROPE_DIGEST, 128, 64, 2, 5003),     # 192 dims
    (synth.MODE_DIGEST, 256, 32, 1, 4000),          # 256 dims (run-time loop only)
    (synth.MODE_ROPE_DIGEST, 64, 16, 2, 262144),    # long spans: many four-tile runs per wave
])
def test_every_key_within_certified_bound(ctx, mode, r, H, B, T):
    """key~ of every archived row against the oracle's exact key, within the
    documented bound E = 2 (n + n/32) 2^-23 max_h ||qt_h|| max_u ||x_u||: a key
    lost, misplaced or mis-computed anywhere in a span would break it."""
    say(f"keys within bound mode={mode} r={r} H={H} B={B} T={T}")
    cfg = synth.CONFIGS["cfg4"].with_(mode=mode, r=r, H=H)
    wl = synth.make_workload(cfg, "cuda", B=B, T=T)
    k = max(1, wl["A"] // 32)
    g, _ = gpu_step(ctx, wl, k=k)
    seqs = list(range(B))
    o, (cache, q_lat, q_rope, P, index, *_rest) = oracle_step(wl, seqs, k=k)
    rr = r if mode != synth.MODE_ROPE else 0
    cols, has_rope = index_cols(mode, r)
    qt, *_ = oracle.query_prep(q_lat, q_rope, P, rr, mode)
    A = wl["A"]
    for j, b in enumerate(seqs):
        x = oracle.index_rows(cache[j], index[j] if index is not None else None, mode, rr, has_rope)
        n = x.shape[1]
        qn = np.linalg.norm(oracle.decode_bf16(qt[j]), axis=1).max()
        xn = np.linalg.norm(oracle.decode_bf16(x[:A]), axis=1).max()
        E = 2 * (n + n / 32) * 2.0 ** -23 * qn * xn
        err = np.abs(g["key"][b, :A].astype(np.float64) - o[b]["key"])
        say(f"  seq {b}: max |key~ - key| {err.max():.3e}, bound {E:.3e}")
        assert np.all(err <= E), (b, int(np.argmax(err)), err.max(), E)
    check_step(wl, g, o, seqs)


@pytest.mark.parametrize("mode,r,H,B,T", [
    (synth.MODE_ROPE_DIGEST, 64, 128, 2, 9000),     # 128 dims, 128 heads: the two-tier shape
    (synth.MODE_ROPE_DIGEST, 128, 64, 2, 5003),     # 192 dims, ragged archive
    (synth.MODE_ROPE_DIGEST, 32, 32, 1, 4000),      # 96 dims, 32 heads
    (synth.MODE_ROPE_DIGEST, 64, 16, 2, 262144),    # long spans: four-tile runs per wave
    (synth.MODE_ROPE_DIGEST, 96, 24, 1, 3001),      # 160 dims; 24 heads in two head tiles (slots repeat heads)
    (synth.MODE_ROPE_DIGEST, 192, 40, 1, 2500),     # 256 dims (run-time loop only), 40 heads
])
def test_every_bound_within_certified_band(ctx, mode, r, H, B, T):
    """UB~ of every archived row against the oracle's exact bound
    UB_u = max_h (s^_h(u) + B_h(u)) (Lemma (Index certificate)), within the
    documented band E + 2^-21 (max |s^| + max_u (amax eta + nmax eps + emax gam))."""
    say(f"bounds within band mode={mode} r={r} H={H} B={B} T={T}")
    cfg = synth.CONFIGS["cfg3"].with_(mode=mode, r=r, H=H)
    wl = synth.make_workload(cfg, "cuda", B=B, T=T)
    k = max(1, wl["A"] // 32)
    g, _ = gpu_step(ctx, wl, k=k, two_tier=True)
    seqs = list(range(B))
    o, (cache, q_lat, q_rope, P, index, eta, eps, gam) = oracle_step(wl, seqs, k=k, two_tier=True)
    cols, has_rope = index_cols(mode, r)
    qt, a, nq, e = oracle.query_prep(q_lat, q_rope, P, r, mode)
    A = wl["A"]
    for j, b in enumerate(seqs):
        x = oracle.index_rows(cache[j], index[j] if index is not None else None, mode, r, has_rope)
        n = x.shape[1]
        ub = oracle.upper_bounds(qt[j], a[j], nq[j], e[j], x, eta[j], eps[j], gam[j], A)
        qn = np.linalg.norm(oracle.decode_bf16(qt[j]), axis=1).max()
        xn = np.linalg.norm(oracle.decode_bf16(x[:A]), axis=1).max()
        E = 2 * (n + n / 32) * 2.0 ** -23 * qn * xn
        f64 = lambda v: np.asarray(v, np.float64)
        bmax = (f64(a[j]).max() * f64(eta[j][:A]) + f64(nq[j]).max() * f64(eps[j][:A])
                + f64(e[j]).max() * f64(gam[j][:A])).max()
        band = E + 2.0 ** -21 * (qn * xn + bmax)
        err = np.abs(g["ub"][b, :A].astype(np.float64) - ub)
        say(f"  seq {b}: max |UB~ - UB| {err.max():.3e}, band {band:.3e}")
        assert np.all(err <= band), (b, int(np.argmax(err)), err.max(), band)
    check_step(wl, g, o, seqs, two_tier=True)


def test_longest_spans_at_256_dims_sampled(ctx):
    """256 index dims (digest r=256): the scorer keeps 64 tiles of keys per
    wave at this width, and B=8, A=262144 gives every wave exactly 64 tiles.
    key~ of the rows of every wave's last tile in the first and last blocks,
    of the archive's last rows and of a strided sample, against the oracle's
    exact keys (index rows built by the oracle for those rows only), each
    within its own bound 2 (n + n/32) 2^-23 max_h ||qt_h|| ||x_u||."""
    say("longest spans at 256 dims, sampled keys")
    cfg = synth.CONFIGS["cfg2_r256"].with_(H=16)
    wl = synth.make_workload(cfg, "cuda", B=8, T=262144 + 256)
    A = wl["A"]
    assert A == 262144
    g, _ = gpu_step(ctx, wl, k=A // 128)
    span = 4 * 16 * 64   # rows of one block: four waves of 64 tiles
    last = np.arange(span - 64, span)
    rows = np.unique(np.concatenate([last, span + last, A - span + last, np.arange(A - 100, A),
                                     np.arange(0, A, 997)]))
    for b in (0, 7):
        cache, q_lat, q_rope, P = host_inputs(wl, [b])
        sub = np.ascontiguousarray(cache[:, rows])
        index, *_ = oracle.digest_build(sub, P, cfg.r, with_rope=False, scalars=False)
        qt, *_ = oracle.query_prep(q_lat, q_rope, P, cfg.r, cfg.mode)
        x = oracle.index_rows(sub[0], index[0], cfg.mode, cfg.r, False)
        key, _ = oracle.index_keys(qt[0], x, len(rows))
        n = x.shape[1]
        qn = np.linalg.norm(oracle.decode_bf16(qt[0]), axis=1).max()
        xn = np.linalg.norm(oracle.decode_bf16(x), axis=1)
        E = 2 * (n + n / 32) * 2.0 ** -23 * qn * xn
        err = np.abs(g["key"][b, rows].astype(np.float64) - key)
        say(f"  seq {b}: {len(rows)} rows, max |key~ - key| / bound {np.max(err / E):.3f}")
        assert np.all(err <= E), (b, int(rows[np.argmax(err / E)]))


def test_longest_spans_two_tier_sampled(ctx):
    """The bound form of the scan at 128 dims keeps keys and bounds of 64
    tiles per wave; B=8, A=262144 gives every wave exactly 64 tiles.  key~
    and UB~ of every wave's last tile in the first and last blocks, of the
    archive's last rows and of a strided sample against the oracle's exact
    key and bound (index rows and row scalars built by the oracle for those
    rows only), each within its own band."""
    say("longest spans, two-tier, sampled keys and bounds")
    cfg = synth.CONFIGS["cfg3"].with_(H=16)
    wl = synth.make_workload(cfg, "cuda", B=8, T=262144 + 256)
    A = wl["A"]
    assert A == 262144
    g, _ = gpu_step(ctx, wl, k=A // 32, two_tier=True)
    span = 4 * 16 * 64   # rows of one block: four waves of 64 tiles
    last = np.arange(span - 64, span)
    rows = np.unique(np.concatenate([last, span + last, A - span + last, np.arange(A - 100, A),
                                     np.arange(0, A, 997)]))
    f64 = lambda v: np.asarray(v, np.float64)
    for b in (0, 7):
        cache, q_lat, q_rope, P = host_inputs(wl, [b])
        sub = np.ascontiguousarray(cache[:, rows])
        index, eta, eps, gam = oracle.digest_build(sub, P, cfg.r, with_rope=True, scalars=True)
        qt, a, nq, e = oracle.query_prep(q_lat, q_rope, P, cfg.r, cfg.mode)
        x = oracle.index_rows(sub[0], index[0], cfg.mode, cfg.r, True)
        key, _ = oracle.index_keys(qt[0], x, len(rows))
        ub = oracle.upper_bounds(qt[0], a[0], nq[0], e[0], x, eta[0], eps[0], gam[0], len(rows))
        n = x.shape[1]
        qn = np.linalg.norm(oracle.decode_bf16(qt[0]), axis=1).max()
        xn = np.linalg.norm(oracle.decode_bf16(x), axis=1)
        E = 2 * (n + n / 32) * 2.0 ** -23 * qn * xn
        bu = f64(a[0]).max() * f64(eta[0]) + f64(nq[0]).max() * f64(eps[0]) + f64(e[0]).max() * f64(gam[0])
        band = E + 2.0 ** -21 * (qn * xn + bu)
        kerr = np.abs(g["key"][b, rows].astype(np.float64) - key)
        uerr = np.abs(g["ub"][b, rows].astype(np.float64) - ub)
        say(f"  seq {b}: {len(rows)} rows, key err / bound {np.max(kerr / E):.3f}, "
            f"UB err / band {np.max(uerr / band):.3f}")
        assert np.all(kerr <= E), (b, int(rows[np.argmax(kerr / E)]))
        assert np.all(uerr <= band), (b, int(rows[np.argmax(uerr / band)]))


def _random_case(seed, long=False):
    """A seeded random step shape: mode, rank, heads, window, context, budget,
    row distribution, and two-tier on or off (orthonormal basis then).  The
    long family takes contexts of 30k..140k rows with at most 32 heads."""
    import random
    rnd = random.Random((5000 if long else 1000) + seed)
    mode = rnd.choice([synth.MODE_ROPE, synth.MODE_DIGEST, synth.MODE_ROPE_DIGEST])
    r = 0 if mode == synth.MODE_ROPE else 32 * rnd.randint(1, 8)
    two_tier = mode == synth.MODE_ROPE_DIGEST and rnd.random() < 0.4
    basis = "none" if r == 0 else ("orthonormal" if two_tier else rnd.choice(["orthonormal", "gaussian"]))
    H = rnd.choice([1, 3, 8, 16, 24, 40, 64, 100, 128])
    if two_tier or long:
        H = min(H, 32 if long else 64)
    W = rnd.choice([1, 16, 64, 256])
    T = W + (rnd.randint(30000, 140000) if long else rnd.randint(1, 12000))
    A = T - W
    k = rnd.choice([0, 1, rnd.randint(1, A), A, max(1, A // 32)])
    cfg = synth.CONFIGS["cfg0"].with_(mode=mode, r=r, basis=basis, H=H, W=W, k=k, T=T,
                                      rows=rnd.choice(["gaussian", "mixture", "lognormal"]),
                                      needles=rnd.randint(0, 8), two_tier=two_tier, seed=77 + seed)
    return cfg, (1 if long else rnd.randint(1, 3))


@pytest.mark.parametrize("seed", list(range(40)))
def test_random_shapes_against_the_oracle(ctx, seed):
    """Seeded random shapes over modes, ranks, head counts, windows, ragged
    contexts, budgets (0, 1, A, random), row distributions and the two-tier
    admission: the whole step on every sequence against the oracle."""
    _check_random_case(ctx, *_random_case(seed), f"random case {seed}")


@pytest.mark.parametrize("seed", list(range(8)))
def test_random_long_contexts_against_the_oracle(ctx, seed):
    """The same over contexts of 30k..140k rows (multi-block counting and
    bracket, unrolled scan runs, many attention splits), one sequence each."""
    _check_random_case(ctx, *_random_case(seed, long=True), f"random long case {seed}")


def _check_random_case(ctx, cfg, B, name):
    say(f"{name}: B={B} {synth.describe(cfg)}")
    wl = synth.make_workload(cfg, "cuda", B=B)
    g, _ = gpu_step(ctx, wl, two_tier=cfg.two_tier)
    seqs = list(range(B))
    o, _ = oracle_step(wl, seqs, two_tier=cfg.two_tier)
    check_step(wl, g, o, seqs, two_tier=cfg.two_tier)


def test_determinism(ctx):
    say("determinism")
    cfg = synth.CONFIGS["cfg3"].with_(H=16)
    wl = synth.make_workload(cfg, "cuda", B=2, T=4000)
    g1, _ = gpu_step(ctx, wl, k=100, two_tier=True)
    g2, _ = gpu_step(ctx, wl, k=100, two_tier=True)
    for key in ("sel", "theta", "out_bits", "lse", "adm_count", "key", "ub"):
        assert np.array_equal(g1[key], g2[key]), key
    for b in range(2):
        m = int(g1["adm_count"][b])
        assert np.array_equal(g1["adm"][b, :m], g2["adm"][b, :m])


def test_score_timing_records_each_step():
    say("score timing events")
    c = vkv.Context(0)
    cfg = synth.CONFIGS["cfg1"].with_(H=16)
    wl = synth.make_workload(cfg, "cuda", B=2, T=3000)
    pack = gpu_index(c, wl, False)
    c.set_timing(True)
    g = [gpu_step(c, wl, k=64, index_pack=pack)[0] for _ in range(3)]
    ms = c.score_timing()
    assert len(ms) == 3 and all(t > 0 for t in ms), ms
    assert c.score_timing() == []
    c.set_timing(False)
    gpu_step(c, wl, k=64, index_pack=pack)
    assert c.score_timing() == []
    for key in ("sel", "theta", "out_bits", "lse"):
        assert np.array_equal(g[0][key], g[2][key]), key
    c.close()


def test_debug_rows_assertion_passes(ctx, monkeypatch):
    say("VKV_DEBUG_ROWS")
    monkeypatch.setenv("VKV_DEBUG_ROWS", "1")
    c = vkv.Context(0)
    cfg = synth.CONFIGS["cfg3"].with_(H=8)
    wl = synth.make_workload(cfg, "cuda", B=2, T=2000)
    g, _ = gpu_step(c, wl, k=64, two_tier=True)
    o, _ = oracle_step(wl, [0, 1], k=64, two_tier=True)
    check_step(wl, g, o, [0, 1], two_tier=True)
    c.close()


def test_argument_errors_leave_outputs_untouched(ctx):
    say("argument errors")
    cfg = synth.CONFIGS["cfg0"].with_(H=4)
    wl = synth.make_workload(cfg, "cuda", T=500)
    index, has_rope, *_ = gpu_index(ctx, wl, False)
    step = vkv.Step(wl["cache"], wl["q_lat"], wl["q_rope"], wl["W"], wl["mode"], wl["r"],
                    index=index, index_has_rope=has_rope, P=wl["P"])
    bufs = vkv.Buffers(step, 10)
    bufs.sel.fill_(-7)
    with pytest.raises(vkv.VkvError) as ei:
        vkv.select(ctx, step, bufs.ws, wl["A"] + 1, bufs.sel, bufs.theta)
    assert ei.value.code == -1
    with pytest.raises(vkv.VkvError) as ei:
        vkv.query_prep(ctx, step, bufs.ws[:128])
    assert ei.value.code == -7
    torch.cuda.synchronize()
    assert torch.all(bufs.sel == -7)


# ------------------------------------------------------- full-size configs

FULL = ["cfg0", "cfg1", "cfg2_r64", "cfg2_r128", "cfg2_r192", "cfg2_r256", "cfg3", "cfg4"]


@pytest.mark.parametrize("name", FULL)
def test_full_config_every_sequence(ctx, name):
    """Each config at its full size, in the bench's launch configuration: the
    selected (and admitted) sets, theta, outputs and lse of every sequence
    against the oracle, which computes each sequence whole."""
    cfg = synth.CONFIGS[name]
    say(f"full-size {synth.describe(cfg)}")
    wl = synth.make_workload(cfg, "cuda")
    g, _ = gpu_step(ctx, wl, two_tier=cfg.two_tier)
    seqs = list(range(wl["B"]))
    for s0 in range(0, len(seqs), 8):
        part = seqs[s0:s0 + 8]
        o, _ = oracle_step(wl, part, two_tier=cfg.two_tier, nthreads=0)
        check_step(wl, g, o, part, two_tier=cfg.two_tier)
        say(f"  sequences {part[0]}..{part[-1]} match")
    if cfg.two_tier:
        frac = [round(float(g["adm_count"][b] / (wl["A"] - wl["k"])), 4) for b in seqs]
        say(f"admitted fraction of non-selected archive rows: {frac}")
    needles = [len(np.intersect1d(g["sel"][b], wl["needles"][b].numpy())) / max(1, len(wl["needles"][b]))
               for b in seqs]
    say(f"needle recall of S (context only): min {min(needles):.3f} mean {np.mean(needles):.3f}")
    del wl
    torch.cuda.empty_cache()


# ------------------------------------------------- boundary contracts

def test_stage_calls_are_idempotent(ctx):
    """One vkv_query_prep + vkv_score, then vkv_select at k1, k2, k1 and
    vkv_admit twice on the same workspace: every call's result equals the
    oracle's, so nothing a call leaves in the workspace leaks into the next."""
    say("idempotent stage calls")
    cfg = synth.CONFIGS["cfg3"].with_(H=32)
    B, T = 3, 20000
    wl = synth.make_workload(cfg, "cuda", B=B, T=T)
    index, has_rope, eta, eps, gam = gpu_index(ctx, wl, True)
    step = vkv.Step(wl["cache"], wl["q_lat"], wl["q_rope"], wl["W"], wl["mode"], wl["r"], index=index,
                    index_has_rope=has_rope, P=wl["P"], eta=eta, eps=eps, gam=gam)
    A = wl["A"]
    k1, k2 = 600, 37
    ws = vkv.alloc_workspace(step, k1, A)
    key = torch.empty(B, A, dtype=torch.float32, device="cuda")
    ub = torch.empty_like(key)
    vkv.query_prep(ctx, step, ws)
    vkv.score(ctx, step, ws, key, ub)
    cache, q_lat, q_rope, P = host_inputs(wl, range(B))
    oidx, oeta, oeps, ogam = oracle.digest_build(cache, P, cfg.r, with_rope=True)
    qt, a, nq, e = oracle.query_prep(q_lat, q_rope, P, cfg.r, cfg.mode)
    xs = [oracle.index_rows(cache[b], oidx[b], cfg.mode, cfg.r, True) for b in range(B)]
    okeys = [oracle.index_keys(qt[b], xs[b], A)[0] for b in range(B)]
    oubs = [oracle.upper_bounds(qt[b], a[b], nq[b], e[b], xs[b], oeta[b], oeps[b], ogam[b], A)
            for b in range(B)]
    sels = {}
    for k in (k1, k2, k1):
        sel = torch.full((B, k), -5, dtype=torch.int32, device="cuda")
        theta = torch.empty(B, dtype=torch.float64, device="cuda")
        vkv.select(ctx, step, ws, k, sel, theta)
        torch.cuda.synchronize()
        for b in range(B):
            osel, oth = oracle.select(okeys[b], k)
            assert np.array_equal(sel[b].cpu().numpy(), osel), (k, b)
            assert theta[b].item() == oth, (k, b)
        sels[k] = (sel, theta)
        say(f"  select k={k} matches")
    sel, theta = sels[k1]
    for rep in range(2):
        adm = torch.full((B, A), -5, dtype=torch.int32, device="cuda")
        cnt = torch.full((B,), -5, dtype=torch.int32, device="cuda")
        vkv.admit(ctx, step, ws, k1, sel, theta, ub, adm, cnt, A)
        torch.cuda.synchronize()
        for b in range(B):
            oadm, ocnt = oracle.admit(oubs[b], sel[b].cpu().numpy(), theta[b].item())
            assert int(cnt[b]) == ocnt, (rep, b, int(cnt[b]), ocnt)
            assert np.array_equal(adm[b, :ocnt].cpu().numpy(), oadm), (rep, b)
        say(f"  admit call {rep} matches")


@pytest.mark.parametrize("cm", [0.25, 0.05, 0.0])
def test_certificate_multiplier_admission(ctx, cm):
    """Eq. (trigger)'s z / sqrt(d_c - r) below 1 (a calibrated trigger): the
    admitted sets stay bit-exact against the oracle at the same multiplier, and
    shrink with it."""
    say(f"cert_mult {cm}")
    cfg = synth.CONFIGS["cfg3"].with_(H=64)
    wl = synth.make_workload(cfg, "cuda", B=2, T=12000)
    g, _ = gpu_step(ctx, wl, k=375, two_tier=True, cert_mult=cm)
    o, _ = oracle_step(wl, [0, 1], k=375, two_tier=True, cert_mult=cm)
    check_step(wl, g, o, [0, 1], two_tier=True)
    say(f"  admitted per sequence: {[int(c) for c in g['adm_count']]} of {wl['A'] - 375}")


def test_admit_with_another_multiplier_than_the_scan(ctx):
    """vkv_score formed UB~ with cert_mult 1, vkv_admit asks for 0.2: the band
    shortcut is skipped and every row outside S is decided on its exact bound,
    so the admitted set is the oracle's at 0.2."""
    say("admit multiplier differs from the scan's")
    cfg = synth.CONFIGS["cfg3"].with_(H=16)
    wl = synth.make_workload(cfg, "cuda", B=2, T=6000)
    g, (step, bufs, _) = gpu_step(ctx, wl, k=180, two_tier=True, cert_mult=1.0)
    vkv.admit(ctx, step, bufs.ws, 180, bufs.sel, bufs.theta, bufs.ub, bufs.adm, bufs.adm_count,
              bufs.cap, None, 0.2)
    torch.cuda.synchronize()
    o, _ = oracle_step(wl, [0, 1], k=180, two_tier=True, cert_mult=0.2)
    for b in range(2):
        cnt = int(bufs.adm_count[b])
        assert cnt == o[b]["adm_count"], (b, cnt, o[b]["adm_count"])
        assert np.array_equal(bufs.adm[b, :cnt].cpu().numpy(), o[b]["adm"])


def test_row_set_checker_fires_on_broken_lists(ctx):
    """The executable row-set invariant (vkv_check_rows, the check
    VKV_DEBUG_ROWS runs inside the calls) accepts a real step's lists and
    refuses each broken form: unsorted, duplicated or out-of-archive selected
    rows, an admitted row that is also selected, unsorted admitted rows and an
    impossible count."""
    say("row-set checker, known-bad lists")
    cfg = synth.CONFIGS["cfg3"].with_(H=8)
    wl = synth.make_workload(cfg, "cuda", B=2, T=3000)
    k = 64
    g, (step, bufs, _) = gpu_step(ctx, wl, k=k, two_tier=True)
    vkv.check_rows(ctx, step, k, bufs.sel, bufs.adm, bufs.adm_count, bufs.cap)
    A = wl["A"]

    def refused(sel=None, adm=None, cnt=None):
        s = bufs.sel.clone() if sel is None else sel
        a = bufs.adm.clone() if adm is None else adm
        c = bufs.adm_count.clone() if cnt is None else cnt
        with pytest.raises(vkv.VkvError) as ei:
            vkv.check_rows(ctx, step, k, s, a, c, bufs.cap)
        assert ei.value.code == -8, ei.value

    s = bufs.sel.clone(); s[1, [5, 6]] = s[1, [6, 5]]; refused(sel=s)
    s = bufs.sel.clone(); s[0, 9] = s[0, 8]; refused(sel=s)
    s = bufs.sel.clone(); s[0, k - 1] = A; refused(sel=s)
    n0 = int(bufs.adm_count[0])
    assert n0 > 2
    a = bufs.adm.clone(); a[0, 0] = bufs.sel[0, 0]; a[0, :n0] = a[0, :n0].sort().values; refused(adm=a)
    a = bufs.adm.clone(); a[0, [0, 1]] = a[0, [1, 0]]; refused(adm=a)
    c = bufs.adm_count.clone(); c[1] = A - k + 1; refused(cnt=c)
