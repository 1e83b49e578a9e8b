"""Kernel-level parity through the C ABI: the bf16 matrix-product kernel and
the causal attention kernel, at small ragged shapes element by element and at
the full 7B-shape launch sizes on sampled outputs computed one by one."""
import numpy as np
import pytest

from gpu_util import bf16_tensor, bf16_values, log
from oracle.forward import causal_attention
from paper_2409_17836_amd import binding as B
from synth.gen import gen_normal

pytestmark = pytest.mark.gpu


def _gemm_case(M, N, K, seed):
    import torch
    a = bf16_values(gen_normal((M, K), seed))
    b = bf16_values(gen_normal((N, K), seed + 1))
    c = B.op_gemm_bf16(bf16_tensor(a), bf16_tensor(b))
    torch.cuda.synchronize()
    return a, b, c


@pytest.mark.parametrize("M,N,K", [(300, 256, 64), (513, 512, 128), (1, 256, 4096),
                                   (1000, 768, 3072), (256, 2304, 768), (257, 256, 320)])
def test_gemm_small_shapes(M, N, K):
    log(f"gemm {M}x{N}x{K}")
    a, b, c = _gemm_case(M, N, K, 11)
    ref = a.astype(np.float64) @ b.astype(np.float64).T
    np.testing.assert_allclose(c.cpu().numpy(), ref, rtol=1e-5, atol=2e-4 * np.sqrt(K))


@pytest.mark.parametrize("N,K", [(12288, 4096), (4096, 4096), (22016, 4096), (4096, 11008),
                                 (32000 - 32000 % 256, 4096)])
def test_gemm_full_7b_shapes_sampled(N, K):
    """M = 8 windows x 4096 tokens; 4096 sampled outputs per shape."""
    M = 32768
    log(f"gemm full {M}x{N}x{K}")
    a, b, c = _gemm_case(M, N, K, 21)
    rng = np.random.default_rng(N + K)
    i = np.concatenate([rng.integers(0, M, 4090), [0, M - 1, 255, 256, 32767, 12345]])
    j = np.concatenate([rng.integers(0, N, 4090), [0, N - 1, 31, 32, 255, 256]])
    import torch
    got = c[torch.from_numpy(i).cuda(), torch.from_numpy(j).cuda()].cpu().numpy()
    ref = np.einsum("nk,nk->n", a[i].astype(np.float64), b[j].astype(np.float64))
    np.testing.assert_allclose(got, ref, rtol=1e-5, atol=2e-4 * np.sqrt(K))


def _attn_inputs(Bn, Hq, Hkv, W, hd, seed):
    q = bf16_values(gen_normal((Bn, Hq, W, hd), seed))
    k = bf16_values(gen_normal((Bn, Hkv, W, hd), seed + 1))
    v = bf16_values(gen_normal((Bn, Hkv, W, hd), seed + 2))
    return q, k, v


def _run_attn(q, k, v):
    """v is given natural [B, Hkv, W, hd]; the kernel takes it transposed."""
    import torch
    vt = np.ascontiguousarray(np.swapaxes(v, 2, 3))
    o = B.op_attention_bf16(bf16_tensor(q), bf16_tensor(k), bf16_tensor(vt))
    torch.cuda.synchronize()
    return o.float().cpu().numpy()


@pytest.mark.parametrize("Hq,Hkv,W,hd", [(4, 4, 64, 128), (4, 2, 200, 64), (8, 1, 256, 128),
                                         (2, 2, 8, 64), (3, 3, 392, 128)])
def test_attention_small(Hq, Hkv, W, hd):
    log(f"attention Hq={Hq} Hkv={Hkv} W={W} hd={hd}")
    Bn = 2
    q, k, v = _attn_inputs(Bn, Hq, Hkv, W, hd, 5)
    o = _run_attn(q, k, v).reshape(Bn, W, Hq * hd)
    for b in range(Bn):
        f = lambda x: np.swapaxes(x[b], 0, 1).astype(np.float64)
        ref = causal_attention(f(q), f(k), f(v))
        np.testing.assert_allclose(o[b], ref, rtol=1e-2, atol=1e-2)


def test_attention_full_7b_shape_sampled():
    """B=8, H=32, W=4096, hd=128: sampled query rows checked one by one."""
    Bn, H, W, hd = 8, 32, 4096, 128
    log("attention full 7B shape")
    q, k, v = _attn_inputs(Bn, H, H, W, hd, 9)
    o = _run_attn(q, k, v).reshape(Bn, W, H, hd)
    rng = np.random.default_rng(3)
    rows = [(0, 0, 0), (7, 31, 4095), (3, 5, 127), (3, 5, 128), (1, 2, 2047), (6, 30, 4000)]
    rows += [tuple(x) for x in np.stack([rng.integers(0, Bn, 10), rng.integers(0, H, 10),
                                         rng.integers(0, W, 10)], 1)]
    for b, h, i in rows:
        kk = k[b, h, :i + 1].astype(np.float64)
        s = kk @ q[b, h, i].astype(np.float64) / np.sqrt(hd)
        p = np.exp(s - s.max())
        ref = (p / p.sum()) @ v[b, h, :i + 1].astype(np.float64)
        np.testing.assert_allclose(o[b, i, h], ref, rtol=1e-2, atol=1e-2, err_msg=str((b, h, i)))


def _silu(x):
    return x / (1.0 + np.exp(-x))


def _blocked_case(kind, M, N, K, seed):
    """The model's blocked-weight product with its fused epilogue; returns
    (A, B, C0 or None, output tensor)."""
    import torch
    a = bf16_values(gen_normal((M, K), seed))
    b = bf16_values(gen_normal((N, K), seed + 1))
    bb = B.op_block_weights(bf16_tensor(b))
    c0 = None
    if kind == "resid":
        c0 = gen_normal((M, N), seed + 2)
        out = B.op_gemm_bf16_blocked(bf16_tensor(a), bb, "resid", out=torch.from_numpy(c0).cuda())
    else:
        out = B.op_gemm_bf16_blocked(bf16_tensor(a), bb, kind)
    torch.cuda.synchronize()
    return a, b, c0, out


def _blocked_check(kind, a_rows, b, c0_rows, got, K):
    acc = a_rows.astype(np.float64) @ b.astype(np.float64).T
    tol = 2e-4 * np.sqrt(K)
    if kind == "store":
        np.testing.assert_allclose(got, acc, rtol=1e-5, atol=tol)
    elif kind == "resid":
        np.testing.assert_allclose(got, c0_rows.astype(np.float64) + acc, rtol=1e-5, atol=tol)
    else:
        # row 64g + t is gate feature 32g + t, row 64g + 32 + t its up row;
        # the kernel rounds silu(gate) * up to bf16 (one ulp = 2^-8 relative)
        g = acc.reshape(acc.shape[0], -1, 2, 32)
        ref = (_silu(g[:, :, 0]) * g[:, :, 1]).reshape(acc.shape[0], -1)
        np.testing.assert_allclose(got, ref, rtol=2.0 ** -8, atol=1e-3 * np.sqrt(K))


@pytest.mark.parametrize("kind", ["store", "resid", "swiglu"])
@pytest.mark.parametrize("M,N,K", [(300, 512, 128), (1000, 768, 3072), (17, 256, 64), (300, 512, 192),
                                   (129, 256, 320), (64, 1024, 448)])
def test_gemm_blocked_small_shapes(kind, M, N, K):
    """Ragged M (partial row tiles) element by element; K from one 64-wide
    k-stage to several (the stage loop, the stage before the last and the
    last take different paths)."""
    log(f"blocked gemm {kind} {M}x{N}x{K}")
    a, b, c0, out = _blocked_case(kind, M, N, K, 41)
    _blocked_check(kind, a, b, c0, out.float().cpu().numpy(), K)


@pytest.mark.parametrize("kind,N,K", [("swiglu", 22016, 4096), ("resid", 4096, 11008),
                                      ("resid", 4096, 4096), ("store", 12288, 4096),
                                      ("store", 32000, 4096)])
def test_gemm_blocked_full_7b_shapes_sampled(kind, N, K):
    """The instantiations the 7B-shape model runs (weights in MFMA blocks;
    operand ring on B for the wide products, on A for the residual adds) at
    M = 8 windows x 4096 tokens: 64 sampled rows, every column."""
    import torch
    M = 32768
    log(f"blocked gemm full {kind} {M}x{N}x{K}")
    a, b, c0, out = _blocked_case(kind, M, N, K, 51)
    rng = np.random.default_rng(N + K)
    rows = np.unique(np.concatenate([rng.integers(0, M, 60), [0, 255, 256, M - 1]]))
    got = out[torch.from_numpy(rows).cuda()].float().cpu().numpy()
    _blocked_check(kind, a[rows], b, None if c0 is None else c0[rows], got, K)
