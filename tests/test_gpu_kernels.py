"""GPU parity of each kernel against the float64 oracle, through the C ABI.

Small shapes span several tiles and ragged tails; full shapes are the 8B-shaped
target / 1B-shaped drafter projections and attention at the verify launch
configuration, checked on sampled outputs the oracle computes one by one.
"""

import numpy as np
import pytest

from oracle import decoder as OD
from oracle import philox as OP
from tests.gpu_util import bf16_bits, device, rel_err, say, torch, widen_bits

pytestmark = pytest.mark.gpu


def B():
    from paper_2607_20507_amd import binding
    return binding


# ---------------------------------------------------------------------------
# Philox

@pytest.mark.parametrize("seed,seq,pos,purpose", [(0, 0, 0, 0), (1234, (1 << 40) + 7, 513, 1),
                                                  ((1 << 64) - 1, 99, 4095, 2), (5, 3, 7, 3)])
def test_philox_uniform_bit_exact(seed, seq, pos, purpose):
    dev = device()
    n = 1003
    out = torch.empty(n, dtype=torch.float32, device=dev)
    say("philox", seed, seq, pos, purpose)
    B().spec_philox_uniform(seed, seq if seq < (1 << 63) else seq - (1 << 64), pos, purpose, n, out)
    torch.cuda.synchronize()
    ref = OP.to_uniform(OP.raw_words(seed, seq, pos, purpose, n))
    assert np.array_equal(out.cpu().numpy().astype(np.float64), ref)


# ---------------------------------------------------------------------------
# GEMM

def _rand_bf16(shape, std, gen_seed, dev):
    g = torch.Generator(device=dev)
    g.manual_seed(gen_seed)
    return (torch.randn(*shape, generator=g, device=dev) * std).to(torch.bfloat16)


def _gemm_case(dt, R, N, K, epi, dev, seed=0, cols=None, splitk=True):
    b = B()
    rows_w = 2 * N if epi == b.SPEC_EPI_SWIGLU else N
    if dt == b.SPEC_BF16:
        X = _rand_bf16((R, K), 1.0, seed + 1, dev)
        W = _rand_bf16((rows_w, K), 0.05, seed + 2, dev)
    else:
        g = torch.Generator(device=dev)
        g.manual_seed(seed + 3)
        X = torch.randn(R, K, generator=g, device=dev)
        W = torch.randn(rows_w, K, generator=g, device=dev) * 0.05
    if epi == b.SPEC_EPI_SWIGLU:
        Y = torch.zeros(R, N, dtype=X.dtype, device=dev)
    elif epi == b.SPEC_EPI_ADD_F32:
        Y = torch.randn(R, N, device=dev)
    else:
        Y = torch.full((R, N), float("nan"), device=dev)
    Y0 = Y.float().cpu().numpy().astype(np.float64)
    Wk = W
    if dt == b.SPEC_BF16:  # the bf16 kernels read the tiled layout (gate and up halves packed separately)
        Wk = W.clone()
        for h in range(rows_w // N):
            b.spec_pack_weight(Wk[h * N:(h + 1) * N], N, K)
    ws = None
    if splitk:
        ws = torch.empty(b.spec_op_gemm_workspace_bytes(R, rows_w), dtype=torch.uint8, device=dev)
    say("gemm", dt, R, N, K, epi, "splitk" if splitk else "")
    b.spec_op_gemm(dt, R, N, K, X, Wk, Y, epi, ws)
    torch.cuda.synchronize()
    if cols is None:
        cols = np.arange(N)
    cols_t = torch.from_numpy(cols).to(dev)
    if dt == b.SPEC_BF16:
        x = widen_bits(bf16_bits(X))
        wg = bf16_bits(W.index_select(0, cols_t))
        wu = bf16_bits(W.index_select(0, cols_t + N)) if epi == b.SPEC_EPI_SWIGLU else None
    else:
        x = X.cpu().numpy().astype(np.float64)
        wg = W.index_select(0, cols_t).cpu().numpy()
        wu = W.index_select(0, cols_t + N).cpu().numpy() if epi == b.SPEC_EPI_SWIGLU else None
    gref = OD.matmul_wt(x, wg)
    got = Y.float().cpu().numpy().astype(np.float64)[:, cols]
    if epi == b.SPEC_EPI_STORE_F32:
        return got, gref
    if epi == b.SPEC_EPI_ADD_F32:
        return got, Y0[:, cols] + gref
    return got, OD.silu(gref) * OD.matmul_wt(x, wu)


EPIS = [0, 1, 2]


def tiled_layout_ref(w, rot_rows=0, hd=0):
    """The tiled weight layout written out on the CPU from its definition:
    rotary heads reordered (tile t = rows 8t..8t+7, hd/2+8t..hd/2+8t+7), then
    in every full 16-row group and 128-column block the 16 x 16 matrix of
    8-element chunks transposed; a trailing partial group stays as is."""
    rows, K = w.shape
    src = w.copy()
    for h0 in range(0, rot_rows, hd or 1):
        order = [(0 if i < 8 else hd // 2) + 8 * t + (i % 8) for t in range(hd // 16) for i in range(16)]
        src[h0:h0 + hd] = w[h0 + np.array(order)]
    out = src.copy()
    for g0 in range(0, rows - rows % 16, 16):
        blk = src[g0:g0 + 16].reshape(16, K // 128, 16, 8)  # [row, block, chunk, 8]
        out[g0:g0 + 16] = blk.transpose(2, 1, 0, 3).reshape(16, K)
    return out


def kv_block_index(hd):
    """Position of (token k, dim d) inside one (page, kv head) block of the
    bf16 KV cache, from the layout's definition: K unit
    ((s*2 + h)*4 + g)*8 + j with c = d // 8, s = c // 4, g = c % 4,
    h = (k // 4) % 2, j = k % 4 + 4 (k // 8); V unit ((d // 16)*2 + k // 8)*16
    + d % 16; 8 elements per unit.  Returns (ik, iv), int64 [16, hd]."""
    k = np.arange(16)[:, None]
    d = np.arange(hd)[None, :]
    c = d // 8
    ik = ((((c // 4) * 2 + (k // 4) % 2) * 4 + c % 4) * 8 + (k % 4 + 4 * (k // 8))) * 8 + d % 8
    iv = (((d // 16) * 2 + k // 8) * 16 + d % 16) * 8 + k % 8
    return ik.astype(np.int64), iv.astype(np.int64)


def test_kv_block_index_is_a_permutation():
    for hd in (64, 128):
        ik, iv = kv_block_index(hd)
        assert np.array_equal(np.sort(ik.ravel()), np.arange(16 * hd))
        assert np.array_equal(np.sort(iv.ravel()), np.arange(16 * hd))


@pytest.mark.parametrize("rows,K,rot_rows,hd", [(32, 256, 0, 0), (40, 384, 0, 0), (7, 128, 0, 0),
                                               (6 * 64 + 24, 256, 4 * 64, 64), (3 * 128, 128, 2 * 128, 128)])
def test_pack_weight_layout(rows, K, rot_rows, hd):
    dev = device()
    w = _rand_bf16((rows, K), 1.0, rows + K, dev)
    ref = tiled_layout_ref(bf16_bits(w), rot_rows, hd)
    say("pack", rows, K, rot_rows, hd)
    B().spec_pack_weight(w, rows, K, rot_rows, hd)
    torch.cuda.synchronize()
    assert np.array_equal(bf16_bits(w), ref)


@pytest.mark.parametrize("R,N,K", [(1, 48, 128), (6, 200, 256), (16, 64, 384), (17, 100, 128), (33, 130, 256),
                                   (48, 96, 512), (64, 64, 128), (65, 300, 256), (130, 260, 384),
                                   (384, 512, 512), (257, 136, 128), (364, 600, 1024), (129, 257, 640),
                                   (1, 48, 1024), (6, 200, 2048), (33, 130, 1024), (64, 64, 768),
                                   (2, 100, 256), (2, 48, 1152)])
@pytest.mark.parametrize("epi", EPIS)
@pytest.mark.parametrize("splitk", [True, False])
def test_gemm_bf16_small(R, N, K, epi, splitk):
    dev = device()
    got, ref = _gemm_case(B().SPEC_BF16, R, N, K, epi, dev, seed=R * 7 + N, splitk=splitk)
    tol = 1e-2 if epi == 2 else 1e-5
    assert rel_err(got, ref) < tol


@pytest.mark.parametrize("R,N,K", [(1, 48, 64), (5, 1376 // 2, 256), (5, 256, 688), (70, 33, 17), (5, 1024, 256)])
@pytest.mark.parametrize("epi", EPIS)
def test_gemm_f32(R, N, K, epi):
    dev = device()
    got, ref = _gemm_case(B().SPEC_F32, R, N, K, epi, dev, seed=R + N)
    assert rel_err(got, ref) < 1e-5


# 8B-shaped target and 1B-shaped drafter projections at verify (R = 6),
# serving-batch verify (R = 384) and draft decode (R = 1) row counts.
FULL = [
    (6, 6144, 4096, 0), (6, 4096, 4096, 1), (6, 14336, 4096, 2), (6, 4096, 14336, 1), (6, 128256, 4096, 0),
    (384, 6144, 4096, 0), (384, 14336, 4096, 2), (384, 4096, 14336, 1), (384, 128256, 4096, 0),
    (1, 3072, 2048, 0), (1, 8192, 2048, 2), (1, 2048, 8192, 1), (64, 128256, 2048, 0),
    (21, 128256, 2048, 0), (48, 8192, 2048, 2), (43, 2048, 8192, 1), (9, 70000, 256, 0),
    # the register-streamed MFMA kernel: the 364-row serving verify and a
    # 2048-row prefill chunk of the gate/up, and ragged shapes (rows not a
    # multiple of 16, a trailing partial W tile, N % 4 != 0 for the LM-head
    # form)
    (364, 14336, 4096, 2), (2048, 14336, 4096, 2), (200, 24600, 256, 2), (177, 65546, 128, 0),
    # its 64-row form (K split, W tiles of 64 / 128 / 256 rows) at the
    # serving draft steps' and the batch-8 verify's row counts, 32-128 rows
    (41, 3072, 2048, 0), (64, 2048, 2048, 1), (96, 8192, 2048, 2), (100, 4096, 14336, 1),
    (78, 6144, 4096, 0), (32, 4096, 14336, 1), (50, 14336, 4096, 2), (120, 4096, 4096, 1),
    (128, 14336, 4096, 2), (70, 2100, 2048, 0), (364, 4096, 4096, 1), (170, 4100, 2048, 1),
]


@pytest.mark.parametrize("R,N,K,epi", FULL)
def test_gemm_bf16_full_shapes_sampled(R, N, K, epi):
    dev = device()
    cols = np.random.default_rng(N + K).choice(N, size=min(N, 192), replace=False)
    cols = np.unique(np.concatenate([cols, np.arange(max(0, N - 20), N)]))  # the ragged tail too
    got, ref = _gemm_case(B().SPEC_BF16, R, N, K, epi, dev, seed=N, cols=cols)
    tol = 1e-2 if epi == 2 else 1e-4
    assert rel_err(got, ref) < tol


# Residual-add projections with a long reduction at 160+ rows split K in the
# register-streamed kernel (the serving verify's down projection), partials
# summed by the fixed-order reduction; a ragged N too.
@pytest.mark.parametrize("R,N,K", [(364, 4096, 14336), (200, 4100, 8192)])
def test_gemm_bf16_split_add_sampled(R, N, K):
    dev = device()
    cols = np.random.default_rng(N + K).choice(N, size=min(N, 192), replace=False)
    cols = np.unique(np.concatenate([cols, np.arange(max(0, N - 20), N)]))
    got, ref = _gemm_case(B().SPEC_BF16, R, N, K, 1, dev, seed=N + 1, cols=cols, splitk=True)
    assert rel_err(got, ref) < 1e-4


# ---------------------------------------------------------------------------
# RMSNorm and RoPE + KV append

@pytest.mark.parametrize("dt,R,d", [(0, 5, 256), (1, 7, 4096), (1, 3, 2048), (0, 1, 96)])
def test_rmsnorm(dt, R, d):
    dev = device()
    b = B()
    g = torch.Generator(device=dev)
    g.manual_seed(d)
    h = torch.randn(R, d, generator=g, device=dev) * 3
    wt = torch.float32 if dt == 0 else torch.bfloat16
    w = (1 + 0.1 * torch.randn(d, generator=g, device=dev)).to(wt)
    y = torch.empty(R, d, dtype=wt, device=dev)
    say("rmsnorm", dt, R, d)
    b.spec_op_rmsnorm(dt, R, d, h, w, 1e-5, y)
    torch.cuda.synchronize()
    wv = w.cpu().numpy() if dt == 0 else widen_bits(bf16_bits(w))
    ref = OD.rms_norm(h.cpu().numpy().astype(np.float64), wv if dt == 0 else wv.astype(np.float32), 1e-5)
    got = y.float().cpu().numpy()
    assert rel_err(got, ref) < (1e-6 if dt == 0 else 5e-3)


@pytest.mark.parametrize("dt,Hq,Hkv,hd,theta", [(0, 4, 4, 64, 1e4), (1, 32, 8, 128, 5e5), (1, 32, 8, 64, 5e5)])
def test_rope_kv_append(dt, Hq, Hkv, hd, theta):
    dev = device()
    b = B()
    R, pages = 9, 12
    rng = np.random.default_rng(hd)
    pos = rng.integers(0, 6000, size=R).astype(np.int32)
    slots = rng.choice(pages * 16, size=R, replace=False).astype(np.int32)
    qkv = torch.from_numpy(rng.standard_normal((R, (Hq + 2 * Hkv) * hd)).astype(np.float32)).to(dev)
    et = torch.float32 if dt == 0 else torch.bfloat16
    q = torch.zeros(R, Hq, hd, dtype=et, device=dev)
    kp = torch.zeros(pages, Hkv, 16, hd, dtype=et, device=dev)
    vp = torch.zeros(pages, Hkv, hd, 16, dtype=et, device=dev)
    say("rope_kv", dt, Hq, Hkv, hd)
    b.spec_op_rope_kv(dt, R, Hq, Hkv, hd, theta, qkv, torch.from_numpy(pos).to(dev),
                      torch.from_numpy(slots).to(dev), q, kp, vp)
    torch.cuda.synchronize()
    x = qkv.cpu().numpy().astype(np.float64)
    qr = OD.rope(x[:, :Hq * hd].reshape(R, Hq, hd), pos, theta)
    kr = OD.rope(x[:, Hq * hd:(Hq + Hkv) * hd].reshape(R, Hkv, hd), pos, theta)
    vr = x[:, (Hq + Hkv) * hd:].reshape(R, Hkv, hd)
    tol = 1e-5 if dt == 0 else 8e-3
    assert rel_err(q.float().cpu().numpy(), qr) < tol
    kpn, vpn = kp.float().cpu().numpy(), vp.float().cpu().numpy()
    ik, iv = kv_block_index(hd)
    for r in range(R):
        pg, off = divmod(int(slots[r]), 16)
        if dt == 0:
            kg, vg = kpn[pg, :, off, :], vpn[pg, :, :, off]
        else:  # bf16 blocks are in the attention operand order
            kg = kpn[pg].reshape(Hkv, 16 * hd)[:, ik[off]]
            vg = vpn[pg].reshape(Hkv, 16 * hd)[:, iv[off]]
        assert rel_err(kg, kr[r]) < tol
        assert rel_err(vg, vr[r]) < tol


# ---------------------------------------------------------------------------
# paged attention

def _attn_case(dt, rows, pos0, Hq, Hkv, hd, seed, check_seqs=None):
    dev = device()
    b = B()
    rng = np.random.default_rng(seed)
    n = len(rows)
    ctx = [p + r for p, r in zip(pos0, rows)]
    max_pages = max((c + 15) // 16 for c in ctx)
    total_pages = sum((c + 15) // 16 for c in ctx)
    perm = rng.permutation(total_pages + 3)
    ptab = np.zeros((n, max_pages), dtype=np.int32)
    et = torch.float32 if dt == 0 else torch.bfloat16
    Kd, Vd = [], []
    kpool = torch.zeros(total_pages + 3, Hkv, 16, hd, dtype=torch.float32, device=dev)
    vpool = torch.zeros(total_pages + 3, Hkv, hd, 16, dtype=torch.float32, device=dev)
    used = 0
    for i in range(n):
        npg = (ctx[i] + 15) // 16
        ptab[i, :npg] = perm[used:used + npg]
        used += npg
        g = torch.Generator(device=dev)
        g.manual_seed(seed * 100 + i)
        K = torch.randn(ctx[i], Hkv, hd, generator=g, device=dev).to(et).float()
        V = torch.randn(ctx[i], Hkv, hd, generator=g, device=dev).to(et).float()
        Kd.append(K.cpu().numpy().astype(np.float64))
        Vd.append(V.cpu().numpy().astype(np.float64))
        pg = torch.from_numpy(ptab[i, :npg].astype(np.int64)).to(dev)
        t = torch.arange(ctx[i], device=dev)
        kpool[pg[t // 16], :, t % 16, :] = K
        vpool.permute(0, 3, 1, 2)[pg[t // 16], t % 16, :, :] = V
    if dt == 1:  # bf16 blocks in the attention operand order
        ik, iv = (torch.from_numpy(a).to(dev) for a in kv_block_index(hd))
        P = kpool.shape[0]
        kt = torch.empty(P, Hkv, 16 * hd, device=dev)
        vt = torch.empty(P, Hkv, 16 * hd, device=dev)
        kt[:, :, ik.reshape(-1)] = kpool.reshape(P, Hkv, 16 * hd)
        vt[:, :, iv.reshape(-1)] = vpool.permute(0, 1, 3, 2).reshape(P, Hkv, 16 * hd)
        kpool, vpool = kt.reshape(P, Hkv, 16, hd), vt.reshape(P, Hkv, hd, 16)
    kpool, vpool = kpool.to(et), vpool.to(et)
    R = sum(rows)
    g = torch.Generator(device=dev)
    g.manual_seed(seed + 999)
    q = torch.randn(R, Hq, hd, generator=g, device=dev).to(et)
    out = torch.full((R, Hq * hd), float("nan"), device=dev).to(et)
    wsb = b.spec_op_attention_workspace_bytes(n, R, max_pages, Hkv, hd)
    ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
    say("attention", dt, rows[:4], pos0[:4], Hq, Hkv, hd)
    b.spec_op_attention(dt, rows, pos0, ptab, Hq, Hkv, hd, q, kpool, vpool, out, ws)
    torch.cuda.synchronize()
    qn = q.float().cpu().numpy().astype(np.float64)
    on = out.float().cpu().numpy()
    worst = 0.0
    r0 = 0
    for i in range(n):
        if check_seqs is None or i in check_seqs:
            qp = np.arange(pos0[i], pos0[i] + rows[i])
            ref = OD.attention(qn[r0:r0 + rows[i]], Kd[i], Vd[i], qp).reshape(rows[i], Hq * hd)
            worst = max(worst, rel_err(on[r0:r0 + rows[i]], ref))
        r0 += rows[i]
    return worst


@pytest.mark.parametrize("dt,rows,pos0,Hq,Hkv,hd", [
    (1, [5, 1, 8], [37, 100, 16], 8, 2, 64),       # GQA verify windows, 2 query tiles
    (1, [6, 6], [20, 300], 4, 4, 64),              # MHA (small bf16 pair shape)
    (1, [70], [0], 32, 8, 128),                    # prefill: causal from position 0, 5 query tiles
    (1, [3, 17], [1, 33], 16, 16, 64),             # rows beyond one tile with G = 1
    (0, [5, 1], [128, 3], 4, 4, 64),               # fp32 path
    (0, [40], [0], 4, 4, 64),
    # the prefill form (every sequence 64+ rows): blocks of 256 / G rows
    # against all their keys, K / V staged in LDS 64 keys at a time
    (1, [300], [0], 32, 8, 64),                    # head dim 64, a ragged last block and stage
    (1, [200, 90], [0, 333], 32, 8, 128),          # two sequences, the second a later chunk
    (1, [256, 70], [5, 0], 16, 16, 64),            # G = 1: 256-row blocks
    (1, [130], [1000], 8, 2, 64),                  # a chunk continuing at position 1000
    (1, [1024], [0], 32, 8, 128),                  # 16 blocks, 16 stages for the last
])
def test_attention_small(dt, rows, pos0, Hq, Hkv, hd):
    err = _attn_case(dt, rows, pos0, Hq, Hkv, hd, seed=sum(rows) + Hq)
    assert err < (1e-5 if dt == 0 else 1.5e-2)


def test_attention_8b_verify_full():
    """8B-shaped target verify: 1 sequence, context 2048, 6 rows (split context)."""
    assert _attn_case(1, [6], [2048], 32, 8, 128, seed=3) < 1.5e-2


def test_attention_serving_batch_sampled():
    """64 sequences, log-uniform contexts in [512, 4096], k in {3,5,7}."""
    from workloads import SERVING_8B, context_lengths_loguniform, draft_lengths
    ctx = context_lengths_loguniform(SERVING_8B.seed, 64, 512, 4096)
    ks = draft_lengths(SERVING_8B.seed, 64, (3, 5, 7))
    err = _attn_case(1, [int(k) + 1 for k in ks], [int(c) for c in ctx], 32, 8, 128, seed=4,
                     check_seqs={0, 17, 40, 63})
    assert err < 1.5e-2


def test_attention_draft_decode():
    """1B-shaped drafter decode: hd 64, GQA 32/8, 1-2 rows per sequence."""
    assert _attn_case(1, [1, 2, 1], [2047, 900, 5], 32, 8, 64, seed=5) < 1.5e-2
