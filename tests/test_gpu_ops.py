"""Stage-level parity of each HIP kernel against the oracle's definition.

Inputs are seeded, rounded to bf16 on the host, and the oracle runs in fp64
on exactly those bf16 values, so the only differences are the kernel's fp32
arithmetic and its bf16 output rounding.
"""
import numpy as np
import pytest

from gpu_util import torch_cuda
from oracle import encoder as E
from paper_2605_01060_amd import surge as S
from paper_2605_01060_amd import workload as W

pytestmark = pytest.mark.gpu

BF16_REL = 2.0 ** -8  # one bf16 ulp relative to the value


def _bf16(torch, a):
    """float array -> (bf16 GPU tensor, fp64 copy of the rounded values)."""
    r = W.round_to_bf16(np.asarray(a, np.float32))
    t = torch.from_numpy(r).to(torch.bfloat16).cuda()
    return t, r.astype(np.float64)


def _f32(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()


def _to_np(t):
    return t.float().cpu().numpy().astype(np.float64)


LINEAR_SHAPES = [
    # (N, K, M) for every projection of the encoder shapes; M ragged
    (384, 128, 1), (128, 128, 129), (512, 128, 1000), (128, 512, 77),       # tiny
    (1152, 384, 130), (384, 384, 257), (1536, 384, 96), (384, 1536, 300),   # MiniLM
    (2304, 768, 255), (768, 768, 128), (3072, 768, 513), (768, 3072, 200),  # bge
    (3072, 1024, 64), (1024, 1024, 100), (4096, 1024, 37), (1024, 4096, 129),  # large
    # one 64-wide K stage (a tile's first stage is also its last), both tile configurations
    (128, 64, 300), (256, 64, 8200),
]


@pytest.mark.parametrize("N,K,M", LINEAR_SHAPES)
@pytest.mark.parametrize("epi", [0, 1, 2])
def test_linear(N, K, M, epi):
    torch = torch_cuda()
    rng = np.random.default_rng(N * 7 + K * 3 + M + epi)
    x, x64 = _bf16(torch, rng.standard_normal((M, K)))
    w, w64 = _bf16(torch, rng.standard_normal((N, K)) * 0.05)  # [out, in]
    b64 = rng.standard_normal(N) * 0.1
    b = _f32(torch, b64)
    b64 = b64.astype(np.float32).astype(np.float64)
    res, r64 = _bf16(torch, rng.standard_normal((M, N)))
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    S.surge_op_linear(M, N, K, x, w, b, res if epi == 2 else None, epi, y)
    ref = E.linear(x64, w64.T, b64)
    if epi == 1:
        ref = E.gelu(ref)
    if epi == 2:
        ref = ref + r64
    got = _to_np(y)
    err = np.abs(got - ref)
    tol = BF16_REL * np.abs(ref) + 1e-3 * np.sqrt(np.mean(ref ** 2))
    assert np.all(err <= tol), (float(err.max()), float((err - tol).max()))


def test_linear_full_chunk_sampled_rows():
    """A 262,144-token chunk through the FFN1 shape of bge (the launch the
    benchmark times), checked on sampled rows including the last one."""
    torch = torch_cuda()
    M, N, K = 262_144, 3072, 768
    g = torch.Generator(device="cuda").manual_seed(0)
    x = torch.randn((M, K), generator=g, device="cuda").to(torch.bfloat16)
    w = (torch.randn((N, K), generator=g, device="cuda") * 0.05).to(torch.bfloat16)
    b = torch.randn((N,), generator=g, device="cuda") * 0.1
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    S.surge_op_linear(M, N, K, x, w, b, None, 1, y)
    rows = np.unique(np.concatenate([np.arange(0, M, 4099), [M - 1, M - 2, 127, 128]]))
    xs = _to_np(x[rows])
    ref = E.gelu(E.linear(xs, _to_np(w).T, b.double().cpu().numpy()))
    got = _to_np(y[rows])
    tol = BF16_REL * np.abs(ref) + 1e-3 * np.sqrt(np.mean(ref ** 2))
    assert np.all(np.abs(got - ref) <= tol)


def _partials(v64, width):
    """Row statistics partials (mean, biased variance) of consecutive
    `width`-feature slices, laid out [part, row, 2] as the kernels expect."""
    M, n = v64.shape
    parts = v64.reshape(M, n // width, width)
    st = np.stack([parts.mean(axis=2), parts.var(axis=2)], axis=2)  # [M, P, 2]
    return np.ascontiguousarray(st.transpose(1, 0, 2))


LN_SHAPES = [  # (N, K, M): small tiles with ragged M, and >= 8192 rows for 256 x 256 tiles
    (2304, 768, 255), (3072, 768, 513), (768, 768, 128), (768, 3072, 200), (1152, 384, 130),
    (768, 768, 9000), (3072, 768, 8193),
    (256, 64, 8200), (128, 64, 77),  # a single K stage per tile
]


@pytest.mark.parametrize("N,K,M", LN_SHAPES)
@pytest.mark.parametrize("epi", [3, 4, 5, 6])
def test_linear_layernorm_fused(N, K, M, epi):
    """The fused forms against the plain definition: LN(x) W^T + b (+GELU)
    for the folded input, x W^T + b + res or + LN(res) with the output's row
    statistics, on sampled rows (all rows when M is small)."""
    torch = torch_cuda()
    rng = np.random.default_rng(N + 3 * K + 7 * M + 11 * epi)
    eps = 1e-12
    x, x64 = _bf16(torch, rng.standard_normal((M, K)) * 1.5 + 0.3)
    w32 = W.round_to_bf16((rng.standard_normal((N, K)) * 0.05).astype(np.float32))
    w64 = w32.astype(np.float64)
    b64 = (rng.standard_normal(N) * 0.1).astype(np.float32).astype(np.float64)
    res, r64 = _bf16(torch, rng.standard_normal((M, N)) * 2.0 - 0.5)
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    fold = epi in (3, 4)
    width_out = S.surge_op_linear_stats_width(M, N)
    stats_out = torch.full((N // width_out, M, 2), float("nan"), device="cuda")
    if fold:
        g64 = (1.0 + 0.1 * rng.standard_normal(K)).astype(np.float32).astype(np.float64)
        be64 = (0.1 * rng.standard_normal(K)).astype(np.float32).astype(np.float64)
        wf = W.round_to_bf16((w32 * g64[None, :].astype(np.float32)).astype(np.float32))
        col_s = wf.astype(np.float64).sum(axis=1)
        # the weight the folded GEMM stands for: W' = W_eff diag(gamma) exactly
        # (bf16(W gamma) differs from W gamma by one rounding; the encoder
        # tests cover that effect end to end)
        w64 = wf.astype(np.float64) / g64[None, :]
        bias = b64 + w64 @ be64
        width_in = S.surge_op_linear_stats_width(M, K)
        st_in = _partials(x64, width_in)
        S.surge_op_linear_ln(M, N, K, x, torch.from_numpy(wf).to(torch.bfloat16).cuda(),
                             _f32(torch, bias), None, epi, _f32(torch, st_in), K // width_in,
                             _f32(torch, col_s), None, None, eps, None, y)
    else:
        g64 = (1.0 + 0.1 * rng.standard_normal(N)).astype(np.float32).astype(np.float64)
        be64 = (0.1 * rng.standard_normal(N)).astype(np.float32).astype(np.float64)
        width_in = S.surge_op_linear_stats_width(M, N)
        st_in = _partials(r64, width_in)
        S.surge_op_linear_ln(M, N, K, x, torch.from_numpy(w32).to(torch.bfloat16).cuda(),
                             _f32(torch, b64), res, epi, _f32(torch, st_in), N // width_in, None,
                             _f32(torch, g64), _f32(torch, be64), eps, stats_out, y)
    rows = np.arange(M) if M <= 600 else np.unique(np.concatenate(
        [np.arange(0, M, 97), [M - 1, M - 2, 255, 256]]))
    got = _to_np(y)[rows]
    if fold:
        ref = E.linear(E.layer_norm(x64[rows], g64, be64, eps), w64.T, b64)
        if epi == 4:
            ref = E.gelu(ref)
    else:
        r = r64[rows] if epi == 5 else E.layer_norm(r64[rows], g64, be64, eps)
        ref = E.linear(x64[rows], w64.T, b64) + r
    err = np.abs(got - ref)
    tol = BF16_REL * np.abs(ref) + 1e-3 * np.sqrt(np.mean(ref ** 2))
    assert np.all(err <= tol), (float(err.max()), float((err - tol).max()))
    if not fold:
        # statistics of the stored (bf16) rows, per partial
        st = stats_out.cpu().numpy().astype(np.float64)[:, rows, :]
        want = _partials(got, width_out)
        scale = np.mean(got ** 2)
        assert np.all(np.abs(st[..., 0] - want[..., 0]) <= 1e-5 * np.sqrt(scale) + 1e-6)
        assert np.all(np.abs(st[..., 1] - want[..., 1]) <= 1e-4 * scale + 1e-6)


@pytest.mark.parametrize("epi,N,K", [(4, 3072, 768), (6, 768, 3072), (3, 2304, 768)])
def test_linear_fused_full_chunk_sampled_rows(epi, N, K):
    """The fused forms at the size the benchmark launches them (a 262,144-row
    chunk of bge: FFN1 with LN1 folded in, FFN2 with the residual LN1 and
    row statistics out, QKV with LN2 folded in), on sampled rows including
    the last ones."""
    torch = torch_cuda()
    M, eps = 262_144, 1e-12
    g = torch.Generator(device="cuda").manual_seed(epi)
    x = (torch.randn((M, K), generator=g, device="cuda") * 1.3 + 0.2).to(torch.bfloat16)
    w = (torch.randn((N, K), generator=g, device="cuda") * 0.05).to(torch.bfloat16)
    b = torch.randn((N,), generator=g, device="cuda") * 0.1
    rows = np.unique(np.concatenate([np.arange(0, M, 4099), [M - 1, M - 2, 255, 256]]))
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    rng = np.random.default_rng(epi)
    if epi in (3, 4):
        x64 = _to_np(x)
        width = S.surge_op_linear_stats_width(M, K)
        st = _partials(x64, width)
        gam = (1.0 + 0.1 * rng.standard_normal(K)).astype(np.float32).astype(np.float64)
        bet = (0.1 * rng.standard_normal(K)).astype(np.float32).astype(np.float64)
        w32 = _to_np(w).astype(np.float32)
        wf = W.round_to_bf16(w32 * gam[None, :].astype(np.float32))
        weff = wf.astype(np.float64) / gam[None, :]
        bias = b.double().cpu().numpy() + weff @ bet
        S.surge_op_linear_ln(M, N, K, x, torch.from_numpy(wf).to(torch.bfloat16).cuda(),
                             _f32(torch, bias), None, epi, _f32(torch, st), K // width,
                             _f32(torch, wf.astype(np.float64).sum(axis=1)), None, None, eps,
                             None, y)
        ref = E.linear(E.layer_norm(x64[rows], gam, bet, eps), weff.T, b.double().cpu().numpy())
        if epi == 4:
            ref = E.gelu(ref)
    else:
        res = (torch.randn((M, N), generator=g, device="cuda") * 1.7 - 0.3).to(torch.bfloat16)
        r64 = _to_np(res)
        width = S.surge_op_linear_stats_width(M, N)
        st = _partials(r64, width)
        gam = (1.0 + 0.1 * rng.standard_normal(N)).astype(np.float32).astype(np.float64)
        bet = (0.1 * rng.standard_normal(N)).astype(np.float32).astype(np.float64)
        stats_out = torch.full((N // width, M, 2), float("nan"), device="cuda")
        S.surge_op_linear_ln(M, N, K, x, w, b, res, epi, _f32(torch, st), N // width, None,
                             _f32(torch, gam), _f32(torch, bet), eps, stats_out, y)
        ref = E.linear(_to_np(x[rows]), _to_np(w).T, b.double().cpu().numpy()) + \
            E.layer_norm(r64[rows], gam, bet, eps)
        got_all = _to_np(y[rows])
        want = _partials(got_all, width)
        so = stats_out.cpu().numpy().astype(np.float64)[:, rows, :]
        scale = np.mean(got_all ** 2)
        assert np.all(np.abs(so[..., 0] - want[..., 0]) <= 1e-5 * np.sqrt(scale) + 1e-6)
        assert np.all(np.abs(so[..., 1] - want[..., 1]) <= 1e-4 * scale + 1e-6)
    got = _to_np(y[rows])
    tol = BF16_REL * np.abs(ref) + 1e-3 * np.sqrt(np.mean(ref ** 2))
    assert np.all(np.abs(got - ref) <= tol)


ATTN_LENGTHS = [1, 2, 3, 4, 15, 16, 17, 31, 32, 33, 63, 64, 65, 127, 128, 129, 255, 256, 511, 512]


@pytest.mark.parametrize("n_heads,d_head", [(2, 64), (4, 32), (12, 32), (12, 64), (16, 64)])
def test_attention_packed_mixed_lengths(n_heads, d_head):
    torch = torch_cuda()
    rng = np.random.default_rng(n_heads * 100 + d_head)
    lengths = list(ATTN_LENGTHS)
    rng.shuffle(lengths)
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    T = int(cu[-1])
    d = n_heads * d_head
    qkv, q64 = _bf16(torch, rng.standard_normal((T, 3 * d)))
    out = torch.full((T, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    S.surge_op_attention(cu, n_heads, d_head, qkv, out)
    got = _to_np(out)
    worst = 0.0
    for i in range(len(lengths)):
        a, b_ = int(cu[i]), int(cu[i + 1])
        ref = E.self_attention(q64[a:b_], n_heads)
        err = np.abs(got[a:b_] - ref)
        tol = BF16_REL * np.abs(ref) + 1.5e-2
        assert np.all(err <= tol), (lengths[i], float(err.max()))
        worst = max(worst, float(err.max()))
    print(f"[attention {n_heads}x{d_head}] max err {worst:.3e}")


@pytest.mark.parametrize("n_heads,d_head", [(12, 64), (12, 32), (4, 32)])
def test_attention_no_cross_text_leak(n_heads, d_head):
    """Texts whose values differ by a large constant: any attention to
    another text would pull outputs away from the text's own value range
    (32-dimensional heads run in adjacent pairs, so this also covers the
    pair path)."""
    torch = torch_cuda()
    rng = np.random.default_rng(5)
    d = n_heads * d_head
    lengths = [40, 70, 33]
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    T = int(cu[-1])
    qkv = rng.standard_normal((T, 3 * d)) * 0.5
    for i, off in enumerate([0.0, 8.0, -8.0]):
        qkv[cu[i]:cu[i + 1], 2 * d:] = off + rng.standard_normal((lengths[i], d)) * 0.1
    t, q64 = _bf16(torch, qkv)
    out = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    S.surge_op_attention(cu, n_heads, d_head, t, out)
    got = _to_np(out)
    for i, off in enumerate([0.0, 8.0, -8.0]):
        blk = got[cu[i]:cu[i + 1]]
        assert np.all(np.abs(blk - off) < 1.0)


@pytest.mark.parametrize("d", [128, 384, 768, 1024])
def test_layernorm(d):
    torch = torch_cuda()
    rng = np.random.default_rng(d)
    M = 1001
    x, x64 = _bf16(torch, rng.standard_normal((M, d)) * 3.0 + 1.5)
    g64 = (1.0 + 0.1 * rng.standard_normal(d)).astype(np.float32).astype(np.float64)
    b64 = (0.1 * rng.standard_normal(d)).astype(np.float32).astype(np.float64)
    y = torch.empty((M, d), dtype=torch.bfloat16, device="cuda")
    S.surge_op_layernorm(M, d, x, _f32(torch, g64), _f32(torch, b64), 1e-12, y)
    ref = E.layer_norm(x64, g64, b64, 1e-12)
    err = np.abs(_to_np(y) - ref)
    assert np.all(err <= BF16_REL * np.abs(ref) + 1e-4), float(err.max())


@pytest.mark.parametrize("d", [128, 384, 768, 1024])
def test_embed_ln(d):
    torch = torch_cuda()
    rng = np.random.default_rng(d + 1)
    vocab, max_pos = 3000, 96
    word, w64 = _bf16(torch, rng.standard_normal((vocab, d)) * 0.02)
    pos, p64 = _bf16(torch, rng.standard_normal((max_pos, d)) * 0.02)
    g64 = (1.0 + 0.02 * rng.standard_normal(d)).astype(np.float32).astype(np.float64)
    b64 = (0.02 * rng.standard_normal(d)).astype(np.float32).astype(np.float64)
    lengths = [1, 2, 7, 33, 64, 95, 96, 5]
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    ids = rng.integers(0, vocab, size=int(cu[-1])).astype(np.int32)
    tok = torch.from_numpy(ids).cuda()
    out = torch.empty((int(cu[-1]), d), dtype=torch.bfloat16, device="cuda")
    S.surge_op_embed_ln(cu, tok, word, vocab, pos, max_pos, _f32(torch, g64), _f32(torch, b64),
                        1e-12, d, out)
    got = _to_np(out)
    wd = {"word_emb": w64, "pos_emb": p64, "ln_e_g": g64, "ln_e_b": b64}
    for i in range(len(lengths)):
        a, b_ = int(cu[i]), int(cu[i + 1])
        ref = E.embed(wd, ids[a:b_].astype(np.int64), 1e-12)
        err = np.abs(got[a:b_] - ref)
        assert np.all(err <= BF16_REL * np.abs(ref) + 1e-4), (i, float(err.max()))


def test_rows_at_the_4096_token_limit():
    """A 4096-token text is 128 blocks of 32 rows, the most a work item's
    7-bit block index holds: embedding and attention (32- and
    64-dimensional heads) must cover every row of it."""
    torch = torch_cuda()
    rng = np.random.default_rng(4096)
    d, vocab, max_pos = 128, 500, 4096
    lengths = [4096, 3, 40]
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    T = int(cu[-1])
    word, w64 = _bf16(torch, rng.standard_normal((vocab, d)) * 0.02)
    pos, p64 = _bf16(torch, rng.standard_normal((max_pos, d)) * 0.02)
    g64 = (1.0 + 0.02 * rng.standard_normal(d)).astype(np.float32).astype(np.float64)
    b64 = (0.02 * rng.standard_normal(d)).astype(np.float32).astype(np.float64)
    ids = rng.integers(0, vocab, size=T).astype(np.int32)
    out = torch.full((T, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    S.surge_op_embed_ln(cu, torch.from_numpy(ids).cuda(), word, vocab, pos, max_pos,
                        _f32(torch, g64), _f32(torch, b64), 1e-12, d, out)
    got = _to_np(out)
    wd = {"word_emb": w64, "pos_emb": p64, "ln_e_g": g64, "ln_e_b": b64}
    for i in range(len(lengths)):
        a, b_ = int(cu[i]), int(cu[i + 1])
        ref = E.embed(wd, ids[a:b_].astype(np.int64), 1e-12)
        assert np.all(np.abs(got[a:b_] - ref) <= BF16_REL * np.abs(ref) + 1e-4), i
    for n_heads, d_head in ((2, 64), (4, 32)):
        qkv, q64 = _bf16(torch, rng.standard_normal((T, 3 * d)))
        att = torch.full((T, d), float("nan"), dtype=torch.bfloat16, device="cuda")
        S.surge_op_attention(cu, n_heads, d_head, qkv, att)
        got = _to_np(att)
        assert not np.isnan(got).any()
        for i in range(len(lengths)):
            a, b_ = int(cu[i]), int(cu[i + 1])
            ref = E.self_attention(q64[a:b_], n_heads)
            err = np.abs(got[a:b_] - ref)
            assert np.all(err <= BF16_REL * np.abs(ref) + 1.5e-2), (n_heads, i, float(err.max()))


def test_embed_ln_reports_out_of_vocab_ids():
    torch = torch_cuda()
    d, vocab, max_pos = 128, 50, 8
    word = torch.zeros((vocab, d), dtype=torch.bfloat16, device="cuda")
    pos = torch.zeros((max_pos, d), dtype=torch.bfloat16, device="cuda")
    g = torch.ones(d, device="cuda")
    b = torch.zeros(d, device="cuda")
    tok = torch.tensor([1, 2, 50, 3], dtype=torch.int32, device="cuda")
    out = torch.empty((4, d), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(S.SurgeError) as ei:
        S.surge_op_embed_ln(np.array([0, 4]), tok, word, vocab, pos, max_pos, g, b, 1e-12, d, out)
    assert ei.value.status == S.SURGE_ERR_INVALID_ARGUMENT


@pytest.mark.parametrize("d", [128, 384, 768, 1024])
def test_pool_l2(d):
    torch = torch_cuda()
    rng = np.random.default_rng(d + 2)
    lengths = [1, 2, 3, 64, 255, 256, 512, 17]
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    x, x64 = _bf16(torch, rng.standard_normal((int(cu[-1]), d)) + 0.3)
    out = torch.full((len(lengths), d), float("nan"), device="cuda")
    S.surge_op_pool_l2(cu, d, x, out)
    got = out.double().cpu().numpy()
    for i in range(len(lengths)):
        ref = E.mean_pool_l2(x64[cu[i]:cu[i + 1]])
        assert np.max(np.abs(got[i] - ref)) < 2e-6, i
