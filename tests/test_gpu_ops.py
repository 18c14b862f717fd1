"""GPU parity of the individual entry points against the oracle (and, for the
plain linear layer, against the definition of the product).

Every case prints its name and sizes before touching the GPU."""
import math
import sys

import numpy as np
import pytest
import torch

from oracle import dard_oracle as O
from paper_2608_26574_amd import dard, synth

pytestmark = pytest.mark.gpu


def announce(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


# ---------------------------------------------------------------- linear
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("M,N,K", [(1, 16, 64), (17, 48, 192), (64, 4096, 4096), (40, 1024, 12288),
                                   (130, 272, 320), (300, 512, 256)])
def test_linear(dtype, M, N, K):
    announce("linear", dtype, M, N, K)
    g = torch.Generator().manual_seed(M * 7 + N)
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    X = torch.randn(M, K, generator=g).to(td)
    W = torch.randn(N, K, generator=g).to(td)
    Y = torch.empty(M, N, device="cuda")
    Wp = torch.empty_like(W).cuda()
    dard.dard_pack_matrix(W.cuda(), Wp)
    dard.dard_linear(X.cuda(), Wp, N, Y)
    torch.cuda.synchronize()
    ref = X.double().numpy() @ W.double().numpy().T
    scale = np.abs(X.double().numpy()) @ np.abs(W.double().numpy()).T
    err = np.abs(Y.cpu().double().numpy() - ref) / (scale + 1e-30)
    assert err.max() < 2e-6, err.max()


# ---------------------------------------------------------------- mask
@pytest.mark.parametrize("B", [1, 5, 32, 63, 64, 65, 128, 129, 200, 256])
@pytest.mark.parametrize("flags", [0, O.F_XSELF_SHADOW, O.F_MKEYS_SHADOW, O.F_C_BIDIR, O.F_ORDER_L2R,
                                   O.F_ORDER_L2R | O.F_XSELF_SHADOW, O.F_C_BIDIR | O.F_MKEYS_SHADOW,
                                   O.F_ORDER_ENTROPY, O.F_ORDER_MARGIN | O.F_FIXED_W])
def test_state_mask_bit_exact(B, flags):
    announce("mask", B, flags)
    b = 3
    rng = np.random.default_rng(B * 3 + flags)
    state = rng.integers(0, 3, (b, B)).astype(np.uint8)
    conf = rng.choice(np.linspace(0.41, 0.89, 7).astype(np.float32), (b, B))   # with ties
    W = (B + 63) // 64
    sel = torch.zeros(b, 2 * B, W, dtype=torch.int64, device="cuda")
    dard.dard_build_state_mask(dev(state), dev(conf), flags, sel)
    torch.cuda.synchronize()
    got = sel.cpu().numpy().view(np.uint64)
    for s in range(b):
        X = O.take_x(state[s], conf[s], flags)
        for r in range(2 * B):
            for j in range(B):
                bit = (int(got[s, r, j // 64]) >> (j % 64)) & 1
                assert bit == int(X[r, j]), (s, r, j)
            for j in range(B, 64 * W):   # unused bits stay clear
                assert ((int(got[s, r, j // 64]) >> (j % 64)) & 1) == 0


# ---------------------------------------------------------------- attention
def _attn_case(b, B, P, Hq, Hkv, dh, dtype, cand_frac, seed, flags=0, cap_extra=3, sample=None):
    """Max |GPU - oracle| over the sequences in `sample` (all by default)."""
    cap = P + 2 * B + cap_extra
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    q, k, v = synth.qkv(b, 2 * B, Hq, Hkv, dh, cap, seed=seed, dtype=td)
    if cand_frac is None:
        _, state, conf = synth.tiny_block(b, B, 100, seed=seed)
    else:
        _, state, conf = synth.workload_block(b, B, cand_frac, 100, seed=seed)
    out = torch.empty_like(q).cuda()
    scale = 1.0 / math.sqrt(dh)
    nws = dard.dard_attention_workspace_bytes(1 if dtype == "bf16" else 0, b, B, Hq, dh, P)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device="cuda")
    # the V operand is dims-major: [b][Hkv][dh][cap]
    dard.dard_masked_attention(q.cuda(), k.cuda(), v.transpose(-1, -2).contiguous().cuda(), P, dev(state), dev(conf),
                               scale, flags, out, ws)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    worst = 0.0
    for s in (range(b) if sample is None else sample):
        qn, kn, vn = q[s].double().numpy(), k[s].double().numpy(), v[s].double().numpy()
        vis = O.visible_keys(state[s], conf[s], P, flags)
        ref = O.masked_attention(qn, kn[:, :P + 2 * B].transpose(1, 0, 2),
                                 vn[:, :P + 2 * B].transpose(1, 0, 2), vis, scale, Hkv)
        worst = max(worst, float(np.max(np.abs(got[s] - ref))))
    return worst


@pytest.mark.parametrize("b", [1, 4, 16])
@pytest.mark.parametrize("frac", [0.1, 0.25, 0.5])
def test_attention_llada_shape(b, frac):
    """The isolated attention workload: 32 heads x 128, prompt 512, block 32."""
    announce("attention 8B-shape", b, frac)
    err = _attn_case(b, 32, 512, 32, 32, 128, "bf16", frac, seed=b * 10 + int(frac * 100))
    assert err < 2e-2, err


@pytest.mark.parametrize("P", [608, 736])
def test_attention_headline_step_prefixes(P):
    """The 8B step's attention at the longer prefixes of its generation (batch 1,
    32 heads x 128, block 32): 11 and 13 key tiles, split 4 and 5 ways."""
    announce("attention 8B step prefix", P)
    err = _attn_case(1, 32, P, 32, 32, 128, "bf16", 0.25, seed=P)
    assert err < 2e-2, err


@pytest.mark.parametrize("P", [832, 928])
def test_attention_multimodal_batch32(P):
    """The multimodal step's attention (batch 32, 32 heads x 128, block 32,
    576 image + 256 text prefix positions and committed blocks), compared on
    sampled sequences (the first, a middle and the last)."""
    announce("attention multimodal batch 32", P)
    err = _attn_case(32, 32, P, 32, 32, 128, "bf16", 0.3, seed=P, sample=(0, 13, 31))
    assert err < 2e-2, err


@pytest.mark.parametrize("P", [1024, 1472])
def test_attention_dream_gqa_shape(P):
    """The 7B GQA attention workload: 28 query heads on 4 KV heads x 128,
    batch 8, block 64, candidate fraction 0.3, prefix of the first and last
    block of a 512-token generation after a 1024-token prompt."""
    announce("attention 7B-GQA-shape", P)
    err = _attn_case(8, 64, P, 28, 4, 128, "bf16", 0.3, seed=P)
    assert err < 2e-2, err


@pytest.mark.parametrize("case", [
    # batch-1 shape (key splits and their merge): scores grow tile by tile
    dict(b=1, B=32, P=736, Hq=4, Hkv=4, profile=(0.05, 1.0, 3.0, 6.0, 10.0)),
    # 7B GQA shape (two key groups merged in the workgroup): large scores first, then small
    dict(b=2, B=64, P=1024, Hq=14, Hkv=2, profile=(10.0, 0.2, 6.0, 0.05)),
    # block keys far above the prefix
    dict(b=2, B=32, P=200, Hq=4, Hkv=2, profile=(0.1, 0.1, 0.1, 0.1, 12.0)),
])
def test_attention_score_jumps(case):
    """Keys scaled tile by tile, so that a row's scores rise far above its
    running maximum in later tiles (by up to 40-70 log2 units): rises of at
    most 8 are taken against the running maximum as it stands, larger ones move
    it.  The outputs must match the oracle as for ordinary inputs."""
    announce("attention score jumps", case)
    b, B, P, Hq, Hkv, dh = case["b"], case["B"], case["P"], case["Hq"], case["Hkv"], 128
    cap = P + 2 * B + 3
    q, k, v = synth.qkv(b, 2 * B, Hq, Hkv, dh, cap, seed=17, dtype=torch.bfloat16)
    prof = case["profile"]
    tile_scale = torch.tensor([prof[(j // 64) % len(prof)] for j in range(cap)], dtype=torch.float32)
    k = (k.float() * tile_scale[None, None, :, None]).bfloat16()
    _, state, conf = synth.workload_block(b, B, 0.3, 100, seed=18)
    out = torch.empty_like(q).cuda()
    scale = 1.0 / math.sqrt(dh)
    ws = torch.empty(max(dard.dard_attention_workspace_bytes(1, b, B, Hq, dh, P), 1), dtype=torch.uint8, device="cuda")
    dard.dard_masked_attention(q.cuda(), k.cuda(), v.transpose(-1, -2).contiguous().cuda(), P, dev(state), dev(conf),
                               scale, 0, out, ws)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    assert np.isfinite(got).all()
    worst, span = 0.0, 0.0
    for s in range(b):
        qn, kn, vn = q[s].double().numpy(), k[s].double().numpy(), v[s].double().numpy()
        vis = O.visible_keys(state[s], conf[s], P, 0)
        ref = O.masked_attention(qn, kn[:, :P + 2 * B].transpose(1, 0, 2), vn[:, :P + 2 * B].transpose(1, 0, 2),
                                 vis, scale, Hkv)
        worst = max(worst, float(np.max(np.abs(got[s] - ref))))
        # spread of the rows' scores in log2 units (how far above a first tile's maximum they rise)
        kk = kn[np.arange(Hq) // (Hq // Hkv), :P + 2 * B]
        sc = np.einsum("rhd,hkd->rhk", qn, kk) * scale / math.log(2)
        span = max(span, float(np.max(sc.max(axis=2) - sc[..., :64].max(axis=2))))
    print(f"score jumps: max |GPU - oracle| {worst:.3e}, scores rise up to {span:.1f} log2 units past the first tile", flush=True)
    assert span > 32.0, span
    assert worst < 2e-2, worst


@pytest.mark.parametrize("case", [
    dict(b=1, B=1, P=0, Hq=2, Hkv=2, dh=128),       # smallest block, no prefix
    dict(b=2, B=5, P=70, Hq=4, Hkv=2, dh=128),      # ragged block, ragged prefix, GQA
    dict(b=1, B=64, P=1024, Hq=7, Hkv=1, dh=128),   # two row tiles, 7:1 GQA
    dict(b=1, B=128, P=33, Hq=2, Hkv=2, dh=128),    # maximum block: 4 row tiles, 2 mask words
    dict(b=3, B=32, P=100, Hq=4, Hkv=4, dh=64),     # head_dim 64
    dict(b=1, B=32, P=4000, Hq=2, Hkv=1, dh=128),   # long prefix: many key splits
    dict(b=2, B=48, P=700, Hq=6, Hkv=2, dh=64),     # head_dim 64, GQA row tiles across heads, key splits
    dict(b=1, B=128, P=2000, Hq=4, Hkv=4, dh=128),  # block 128 with key splits
    dict(b=1, B=256, P=100, Hq=2, Hkv=1, dh=128),   # maximum block: 8 block tiles, 4 mask words
    dict(b=2, B=200, P=64, Hq=4, Hkv=2, dh=64),     # ragged block straddling mask words
])
def test_attention_edges_bf16(case):
    announce("attention edge bf16", case)
    err = _attn_case(case["b"], case["B"], case["P"], case["Hq"], case["Hkv"], case["dh"], "bf16", None, seed=7)
    assert err < 2e-2, err


@pytest.mark.parametrize("flags", [O.F_XSELF_SHADOW, O.F_MKEYS_SHADOW, O.F_C_BIDIR, O.F_ORDER_L2R])
def test_attention_flags_bf16(flags):
    announce("attention flags", flags)
    err = _attn_case(2, 16, 40, 4, 4, 128, "bf16", None, seed=9, flags=flags)
    assert err < 2e-2, err


@pytest.mark.parametrize("flags", [O.F_C_BIDIR, O.F_ORDER_L2R, O.F_ORDER_L2R | O.F_XSELF_SHADOW])
def test_attention_orderings_8b_shape(flags):
    """Candidate-ordering variants (Sec. 5.1) at the 8B shape, batch 4,
    half the block candidates: the mask differs from the primary one in most
    candidate rows."""
    announce("attention ordering 8B-shape", flags)
    err = _attn_case(4, 32, 512, 32, 32, 128, "bf16", 0.5, seed=21 + flags, flags=flags)
    assert err < 2e-2, err


@pytest.mark.parametrize("flags", [O.F_C_BIDIR, O.F_ORDER_L2R])
def test_attention_orderings_f32(flags):
    announce("attention ordering f32", flags)
    err = _attn_case(2, 7, 9, 4, 2, 128, "f32", None, seed=5, flags=flags)
    assert err < 1e-4, err


@pytest.mark.parametrize("case", [dict(b=1, B=32, P=64, Hq=4, Hkv=4, dh=64),
                                  dict(b=2, B=7, P=9, Hq=4, Hkv=2, dh=128),
                                  dict(b=1, B=3, P=0, Hq=1, Hkv=1, dh=64)])
def test_attention_f32(case):
    announce("attention f32", case)
    err = _attn_case(case["b"], case["B"], case["P"], case["Hq"], case["Hkv"], case["dh"], "f32", None, seed=3)
    assert err < 1e-4, err


# ---------------------------------------------------------------- confidence
def _conf_ref(ls, lx=None, w=None, cur=None):
    rows = ls.shape[0]
    am = np.zeros(rows, dtype=np.int64)
    mp = np.zeros(rows)
    pc = np.zeros(rows)
    for r in range(rows):
        row = ls[r] if lx is None else O.mix_logits(lx[r], ls[r], w[r])
        am[r], mp[r], pc[r] = O.confidence(row, None if cur is None else int(cur[r]))
    return am, mp, pc


@pytest.mark.parametrize("rows,V", [(5, 126464), (3, 152064), (7, 2048), (4, 10), (2, 8195), (1, 1)])
def test_confidence_plain(rows, V):
    announce("confidence", rows, V)
    g = torch.Generator().manual_seed(V + rows)
    ld = (V + 3) // 4 * 4
    ls = (torch.randn(rows, ld, generator=g) * 3).float()
    # plant equal maxima in different chunks: the lower index must win
    if V > 9000:
        ls[0, 9000] = 50.0
        ls[0, 100] = 50.0
    cur = torch.randint(0, V, (rows,), generator=g, dtype=torch.int32)
    am = torch.empty(rows, dtype=torch.int32, device="cuda")
    mp = torch.empty(rows, device="cuda")
    pc = torch.empty(rows, device="cuda")
    ws = torch.empty(dard.dard_confidence_workspace_bytes(rows, V), dtype=torch.uint8, device="cuda")
    ls_d = ls.cuda()
    L = dard.lib()
    dard._check(L.dard_confidence(ls_d.data_ptr(), None, None, cur.cuda().data_ptr(), rows, V, ld,
                                  am.data_ptr(), mp.data_ptr(), pc.data_ptr(), None, None, ws.data_ptr(),
                                  ws.numel(),
                                  torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    ram, rmp, rpc = _conf_ref(ls[:, :V].numpy(), cur=cur.numpy())
    assert np.array_equal(am.cpu().numpy(), ram)
    assert np.max(np.abs(mp.cpu().numpy() - rmp) / rmp) < 1e-5
    assert np.max(np.abs(pc.cpu().numpy() - rpc) / np.maximum(rpc, 1e-30)) < 1e-4
    if V > 9000:
        assert am[0].item() == 100


@pytest.mark.parametrize("wvals", [[0.0, 0.3, 1.0, 0.97, 0.05]])
def test_confidence_mixed(wvals):
    announce("confidence mixed", wvals)
    rows, V = len(wvals), 126464
    g = torch.Generator().manual_seed(11)
    ls = torch.randn(rows, V, generator=g) * 2
    lx = torch.randn(rows, V, generator=g) * 2
    w = torch.tensor(wvals, dtype=torch.float32)
    am = torch.empty(rows, dtype=torch.int32, device="cuda")
    mp = torch.empty(rows, device="cuda")
    ws = torch.empty(dard.dard_confidence_workspace_bytes(rows, V), dtype=torch.uint8, device="cuda")
    dard.dard_confidence(ls.cuda(), am, mp, logits_x=lx.cuda(), w=w.cuda(), ws=ws)
    torch.cuda.synchronize()
    ram, rmp, _ = _conf_ref(ls.numpy(), lx.numpy(), w.numpy())
    assert np.array_equal(am.cpu().numpy(), ram)
    assert np.max(np.abs(mp.cpu().numpy() - rmp) / rmp) < 1e-5


def _mix_tie_pair(w, seed=0):
    """Two (x, s) logit pairs whose mixtures (w x) + ((1 - w) s), each product
    and the sum rounded separately in float32 (Eq. 7 as the library states
    it), are equal, while a fused multiply-add w x + round((1 - w) s) makes
    the second one larger.  Found by search on the CPU."""
    rng = np.random.default_rng(seed)
    w = np.float32(w)
    omw = np.float32(1) - w
    x = (rng.standard_normal(200000) * 4).astype(np.float32)
    s = (rng.standard_normal(200000) * 4).astype(np.float32)
    sep = (w * x) + (omw * s)
    fused = (np.float64(w) * x + (omw * s).astype(np.float64)).astype(np.float32)
    order = np.argsort(sep, kind="stable")
    for a in range(len(order) - 1):
        i, j = order[a], order[a + 1]
        if sep[i] == sep[j] and fused[i] != fused[j]:
            lo, hi = (i, j) if fused[i] < fused[j] else (j, i)
            return (x[lo], s[lo]), (x[hi], s[hi])
    raise AssertionError("no pair found")


def test_confidence_mixing_rounds_each_product():
    """Eq. 7 evaluated with every operation rounded once: on a planted tie of
    the separately rounded mixtures the lower index wins; a kernel that fused
    a product into the sum would pick the higher one."""
    announce("confidence mixing rounding")
    V, w = 4096, 0.3
    (x0, s0), (x1, s1) = _mix_tie_pair(w)
    ls = np.full((1, V), -30.0, dtype=np.float32)
    lx = np.full((1, V), -30.0, dtype=np.float32)
    lx[0, 1000], ls[0, 1000] = x0, s0
    lx[0, 3000], ls[0, 3000] = x1, s1
    am = torch.empty(1, dtype=torch.int32, device="cuda")
    mp = torch.empty(1, device="cuda")
    ws = torch.empty(dard.dard_confidence_workspace_bytes(1, V), dtype=torch.uint8, device="cuda")
    dard.dard_confidence(dev(ls), am, mp, logits_x=dev(lx), w=dev(np.array([w], dtype=np.float32)), ws=ws)
    torch.cuda.synchronize()
    assert O.confidence(O.mix_logits(lx[0], ls[0], w))[0] == 1000
    assert am.item() == 1000


@pytest.mark.parametrize("rows,V,mixed", [(5, 126464, False), (3, 152064, False), (4, 2048, False),
                                          (3, 10, False), (2, 8195, False), (1, 1, False), (5, 126464, True),
                                          (3, 9000, True)])
def test_confidence_entropy_margin(rows, V, mixed):
    """Entropy and margin of each (mixed) row, the scores of the entropy and
    margin orderings (Sec. 5.1), against the oracle's float64 definitions,
    with the top-1 statistics of the same launch unchanged."""
    announce("confidence entropy/margin", rows, V, mixed)
    g = torch.Generator().manual_seed(V * 3 + rows)
    ld = (V + 3) // 4 * 4
    ls = (torch.randn(rows, ld, generator=g) * 3).float()
    lx = (torch.randn(rows, ld, generator=g) * 3).float() if mixed else None
    # sharp rows, flat rows and a tie at the top
    ls[0, :V] *= 0.01
    if rows > 1:
        ls[1, V // 2] = 40.0
    if rows > 2 and V > 4:
        ls[2, 1] = ls[2, V - 1] = 30.0
        if mixed:
            lx[2, 1] = lx[2, V - 1] = 30.0
    w = torch.linspace(0.0, 1.0, rows) if mixed else None
    am = torch.empty(rows, dtype=torch.int32, device="cuda")
    mp = torch.empty(rows, device="cuda")
    ent = torch.empty(rows, device="cuda")
    mrg = torch.empty(rows, device="cuda")
    ws = torch.empty(dard.dard_confidence_workspace_bytes(rows, V), dtype=torch.uint8, device="cuda")
    # V columns in rows of ld elements: the padding is never read
    ls_d = ls.cuda()
    lx_d = None if lx is None else lx.cuda()
    w_d = None if w is None else w.cuda()
    ptr = lambda t: None if t is None else t.data_ptr()
    dard._check(dard.lib().dard_confidence(ls_d.data_ptr(), ptr(lx_d), ptr(w_d), None, rows, V, ld,
                                           am.data_ptr(), mp.data_ptr(), None, ent.data_ptr(), mrg.data_ptr(),
                                           ws.data_ptr(), ws.numel(), torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    lsn = ls[:, :V].numpy()
    lxn = None if lx is None else lx[:, :V].numpy()
    ram, rmp, _ = _conf_ref(lsn, lxn, None if w is None else w.numpy())
    assert np.array_equal(am.cpu().numpy(), ram)
    assert np.max(np.abs(mp.cpu().numpy() - rmp) / rmp) < 1e-5
    for r in range(rows):
        row = lsn[r] if lxn is None else O.mix_logits(lxn[r], lsn[r], w[r].item())
        H, m = O.entropy_margin(row)
        assert abs(ent[r].item() - H) <= 1e-4 + 1e-5 * H, (r, ent[r].item(), H)
        assert abs(mrg[r].item() - m) <= 1e-6 + 1e-5 * m, (r, mrg[r].item(), m)
    if rows > 2 and V > 4:
        assert mrg[2].item() == 0.0


# ---------------------------------------------------------------- decisions
def _params(flags=0, tc=0.4, tu=0.9):
    return dict(tau_c=tc, tau_u=tu, lam=O.LAMBDA_DEFAULT, p0=0.1, mask_id=999, flags=flags)


@pytest.mark.parametrize("B", [1, 7, 32, 128, 256])
@pytest.mark.parametrize("flags,tc,tu", [(0, 0.4, 0.9), (O.F_VERIFY_PCUR, 0.3, 0.7), (0, 0.9, 0.9),
                                         (O.F_PROGRESS, 0.4, 1.0), (O.F_PROGRESS | O.F_VERIFY_PCUR, 0.3, 0.7)])
def test_commit_remask_bit_exact(B, flags, tc, tu):
    announce("commit/remask", B, flags, tc, tu)
    b = 4
    rng = np.random.default_rng(B + int(tc * 10))
    p = _params(flags, tc, tu)
    state = rng.integers(0, 3, (b, B)).astype(np.uint8)
    # confidences including the exact threshold values and their neighbours
    pool = np.array([0.0, tc, np.nextafter(np.float32(tc), np.float32(1)), 0.5, tu,
                     np.nextafter(np.float32(tu), np.float32(1)), 0.99, 1.0], dtype=np.float32)
    mp_s = rng.choice(pool, (b, B)).astype(np.float32)
    pc_s = rng.choice(pool, (b, B)).astype(np.float32)
    mp_mix = rng.choice(pool, (b, B)).astype(np.float32)
    am_s = rng.integers(0, 998, (b, B)).astype(np.int32)
    am_mix = rng.integers(0, 998, (b, B)).astype(np.int32)
    cp = dard.make_params(tc, tu, O.LAMBDA_DEFAULT, 0.1, 999, flags)
    w = torch.empty(b, B, device="cuda")
    dard.dard_commit_remask(dard.PHASE_VERIFY, cp, dev(state), maxprob_s=dev(mp_s), pcur_s=dev(pc_s), w_out=w)
    so = torch.empty(b, B, dtype=torch.uint8, device="cuda")
    to = torch.empty(b, B, dtype=torch.int32, device="cuda")
    co = torch.empty(b, B, device="cuda")
    bd = torch.empty(b, dtype=torch.int32, device="cuda")
    dard.dard_commit_remask(dard.PHASE_FINAL, cp, dev(state), dev(mp_s), dev(pc_s), dev(am_s), dev(mp_mix),
                            dev(am_mix), None, so, to, co, bd)
    torch.cuda.synchronize()
    c_sh = pc_s if flags & O.F_VERIFY_PCUR else mp_s
    for s in range(b):
        _, _, _, rw = O.verify_candidates(state[s], c_sh[s], p)
        assert np.array_equal(w[s].cpu().numpy().astype(np.float64), rw), s
        c = np.where(state[s] == O.STATE_M, mp_mix[s], c_sh[s])
        xh = np.where(state[s] == O.STATE_M, am_mix[s], am_s[s])
        st, tk, cf, done = O.finalize(c, xh, p, state[s])
        assert np.array_equal(so[s].cpu().numpy(), st)
        assert np.array_equal(to[s].cpu().numpy(), tk)
        assert np.array_equal(co[s].cpu().numpy(), cf.astype(np.float32))
        assert bd[s].item() == done


@pytest.mark.parametrize("B", [7, 32, 128])
@pytest.mark.parametrize("flags,wf", [(O.F_FIXED_W, 0.0), (O.F_FIXED_W, 0.5), (O.F_FIXED_W, 1.0),
                                      (O.F_ORDER_ENTROPY, 0.0), (O.F_ORDER_MARGIN | O.F_FIXED_W, 0.25)])
def test_commit_remask_variants_bit_exact(B, flags, wf):
    """Fixed guidance weight and the carried key of the entropy / margin
    orderings (Sec. 5.1) through the per-position entry point."""
    announce("commit/remask variants", B, flags, wf)
    b, tc, tu = 3, 0.4, 0.9
    rng = np.random.default_rng(B * 5 + flags)
    p = dict(_params(flags, tc, tu), w_fixed=wf)
    state = rng.integers(0, 3, (b, B)).astype(np.uint8)
    pool = np.array([0.0, tc, 0.5, tu, 0.99, 1.0], dtype=np.float32)
    mp_s = rng.choice(pool, (b, B)).astype(np.float32)
    mp_mix = rng.choice(pool, (b, B)).astype(np.float32)
    am_s = rng.integers(0, 998, (b, B)).astype(np.int32)
    am_mix = rng.integers(0, 998, (b, B)).astype(np.int32)
    key_s = rng.standard_normal((b, B)).astype(np.float32)
    key_mix = rng.standard_normal((b, B)).astype(np.float32)
    cp = dard.make_params(tc, tu, O.LAMBDA_DEFAULT, 0.1, 999, flags, wf)
    w = torch.empty(b, B, device="cuda")
    dard.dard_commit_remask(dard.PHASE_VERIFY, cp, dev(state), maxprob_s=dev(mp_s), w_out=w)
    so = torch.empty(b, B, dtype=torch.uint8, device="cuda")
    to = torch.empty(b, B, dtype=torch.int32, device="cuda")
    co = torch.empty(b, B, device="cuda")
    dard.dard_commit_remask(dard.PHASE_FINAL, cp, dev(state), dev(mp_s), None, dev(am_s), dev(mp_mix),
                            dev(am_mix), None, so, to, co, None, key_s=dev(key_s), key_mix=dev(key_mix))
    torch.cuda.synchronize()
    for s in range(b):
        _, _, _, rw = O.verify_candidates(state[s], mp_s[s], p)
        assert np.array_equal(w[s].cpu().numpy().astype(np.float64), rw), s
        c = np.where(state[s] == O.STATE_M, mp_mix[s], mp_s[s])
        xh = np.where(state[s] == O.STATE_M, am_mix[s], am_s[s])
        st, tk, cf, _ = O.finalize(c, xh, p, state[s])
        assert np.array_equal(so[s].cpu().numpy(), st)
        assert np.array_equal(to[s].cpu().numpy(), tk)
        if flags & (O.F_ORDER_ENTROPY | O.F_ORDER_MARGIN):
            key = np.where(state[s] == O.STATE_M, key_mix[s], key_s[s])
        else:
            key = cf.astype(np.float32)
        assert np.array_equal(co[s].cpu().numpy(), key)


def test_check_states():
    """dard_check_states counts the codes outside {0, 1, 2} and finds the first."""
    announce("state-code check")
    st = torch.tensor([0, 1, 2, 2, 1, 0, 3, 0, 7, 2], dtype=torch.uint8, device="cuda")
    status = torch.full((2,), 99, dtype=torch.int32, device="cuda")
    dard.dard_check_states(st, status)
    assert status.cpu().tolist() == [2, 6]
    st = torch.randint(0, 3, (5000,), dtype=torch.uint8, device="cuda")
    dard.dard_check_states(st, status)
    assert status.cpu().tolist() == [0, -1]
    st[4097] = 255
    st[4999] = 3
    dard.dard_check_states(st, status)
    assert status.cpu().tolist() == [2, 4097]


# ---------------------------------------------------------------- FP8 KV cache
def fp8_codes(x):
    """OCP FP8 E4M3 codes (uint8) of the values O.to_fp8 rounds x to."""
    r = O.to_fp8(x)
    code = np.searchsorted(O.E4M3_VALUES, np.abs(r)).astype(np.uint8)
    return code | np.where(r < 0, 0x80, 0).astype(np.uint8)


def _attn_case_fp8(b, B, P, Hq, Hkv, dh, cand_frac, seed, cap_extra=3):
    """bf16 Q against K and V held as E4M3 codes (DARD_DTYPE_BF16_KV_FP8); the
    reference attends over the codes' values in float64."""
    cap = P + 2 * B + cap_extra
    q, k, v = synth.qkv(b, 2 * B, Hq, Hkv, dh, cap, seed=seed, dtype=torch.bfloat16)
    kc = fp8_codes(k.double().numpy())
    vc = fp8_codes(v.double().numpy())
    kf, vf = O.to_fp8(k.double().numpy()), O.to_fp8(v.double().numpy())
    if cand_frac is None:
        _, state, conf = synth.tiny_block(b, B, 100, seed=seed)
    else:
        _, state, conf = synth.workload_block(b, B, cand_frac, 100, seed=seed)
    out = torch.empty(q.shape, dtype=torch.bfloat16, device="cuda")
    scale = 1.0 / math.sqrt(dh)
    ws = torch.empty(max(dard.dard_attention_workspace_bytes(dard.DTYPE_BF16_KV_FP8, b, B, Hq, dh, P), 1),
                     dtype=torch.uint8, device="cuda")
    dard.dard_masked_attention(q.cuda(), dev(kc), dev(np.ascontiguousarray(vc.transpose(0, 1, 3, 2))), P, dev(state),
                               dev(conf), scale, 0, out, ws)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    qn = q.double().numpy()
    worst = 0.0
    for s in range(b):
        vis = O.visible_keys(state[s], conf[s], P)
        ref = O.masked_attention(qn[s], kf[s, :, :P + 2 * B].transpose(1, 0, 2),
                                 vf[s, :, :P + 2 * B].transpose(1, 0, 2), vis, scale, Hkv)
        worst = max(worst, float(np.max(np.abs(got[s] - ref))))
    return worst


@pytest.mark.parametrize("case", [
    dict(b=1, B=32, P=512, Hq=32, Hkv=32, dh=128, frac=0.25),   # 8B MHA, batch 1 (key splits)
    dict(b=4, B=32, P=512, Hq=32, Hkv=32, dh=128, frac=0.1),    # batch 4 (two key groups)
    dict(b=16, B=32, P=512, Hq=32, Hkv=32, dh=128, frac=0.5),   # batch 16
    dict(b=8, B=64, P=1024, Hq=28, Hkv=4, dh=128, frac=0.3),    # 7B GQA (one key group with fp8)
    dict(b=2, B=5, P=70, Hq=4, Hkv=2, dh=128, frac=None),       # ragged block and prefix: unaligned V chunks
    dict(b=3, B=32, P=100, Hq=4, Hkv=4, dh=64, frac=None),      # head_dim 64
    dict(b=1, B=256, P=100, Hq=2, Hkv=1, dh=128, frac=None),    # maximum block
])
def test_attention_fp8_kv(case):
    announce("attention fp8 kv", case)
    err = _attn_case_fp8(case["b"], case["B"], case["P"], case["Hq"], case["Hkv"], case["dh"], case["frac"], seed=9)
    assert err < 2e-2, err
