"""Kernel-level parity of the HIP path against the oracle's definitions.

Each case calls one kernel through the C ABI (``include/t2i_ops.h``) on
seeded bf16/fp32 inputs and compares with the oracle computing the same
operation in float64 from the same (bf16-rounded) values."""
import ctypes as C

import numpy as np
import pytest
import torch

import synth
import paper_2607_26566_amd as t2i
from paper_2607_26566_amd import _lib
from oracle import dit
from gpu_common import DEV, rel_l2, say, to_dev, to_host

pytestmark = pytest.mark.gpu


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def rnd(seed, shape, std=1.0, bf=True):
    a = synth.normal(seed, (7,), shape, std)
    return synth.round_bf16(a) if bf else a


def run_linear(dtype, epi, A, W, b, resid=None, gate=None, with_copy=False):
    lib = t2i.load()
    M, K = A.shape
    N = W.shape[0]
    dt = "bf16" if dtype == _lib.T2I_BF16 else "f32"
    dA, dW, db = to_dev(A, dt), to_dev(W, dt), to_dev(b, dt)
    out = torch.zeros((M, N), dtype=dA.dtype, device=DEV)
    dR = torch.from_numpy(resid.astype(np.float32)).to(DEV) if resid is not None else None
    dC = torch.zeros((M, N), dtype=torch.bfloat16, device=DEV) if with_copy else None
    dG = torch.from_numpy(gate.astype(np.float32)).to(DEV) if gate is not None else None
    st = lib.t2i_op_linear(dtype, epi, M, N, K, dA.data_ptr(), K, dW.data_ptr(), K, db.data_ptr(),
                           out.data_ptr(), N, dR.data_ptr() if dR is not None else None, N,
                           dC.data_ptr() if dC is not None else None,
                           dG.data_ptr() if dG is not None else None, _stream())
    _lib.check(st)
    torch.cuda.synchronize()
    return out, dR, dC


GEMM_SHAPES = [(300, 192, 128), (1000, 1152, 1152), (64, 3456, 1152), (8192, 1152, 4608),
               (129, 4608, 1152), (240, 2304, 1152), (1, 128, 64), (4096, 3456, 1152),
               (3000, 1296, 1152), (2100, 200, 128), (2100, 202, 64), (8192, 4608, 1152),
               (1900, 4608, 1152), (2000, 4096, 128)]


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
def test_linear_bf16_store_and_gelu(M, N, K):
    say(f"linear bf16 {M}x{N}x{K}")
    A, W, b = rnd(1, (M, K)), rnd(2, (N, K), 0.05), rnd(3, (N,), 0.1)
    ref = dit.linear(A.astype(np.float64), W.astype(np.float64), b.astype(np.float64))
    out, _, _ = run_linear(_lib.T2I_BF16, _lib.T2I_EPI_STORE, A, W, b)
    assert rel_l2(to_host(out), ref) < 3e-3
    out, _, _ = run_linear(_lib.T2I_BF16, _lib.T2I_EPI_GELU, A, W, b)
    assert rel_l2(to_host(out), dit.gelu_tanh(ref)) < 3e-3


def test_linear_bf16_tilings_agree_bitwise():
    """The same rows through the three GEMM kernels -- direct-load 256-row
    tiles (2100 rows), register-staged 128 x 144 tiles (1900 rows) and 64 x 64
    tiles (300 rows) -- come out bitwise equal: every kernel accumulates K in
    the same order, which is what makes a packed batch equal its requests run
    alone."""
    N, K = 4608, 1152
    A, W, b = rnd(70, (2100, K)), rnd(71, (N, K), 0.05), rnd(72, (N,), 0.1)
    outs = []
    for M in (2100, 1900, 300):
        out, _, _ = run_linear(_lib.T2I_BF16, _lib.T2I_EPI_GELU, A[:M], W, b)
        outs.append(to_host(out)[:300])
    say(f"tilings: max |diff| {np.abs(outs[0] - outs[1]).max():.1e}, {np.abs(outs[0] - outs[2]).max():.1e}")
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


@pytest.mark.parametrize("M,N,K", [(300, 192, 128), (1000, 1152, 4608), (8192, 1152, 1152),
                                   (4096, 2304, 1152), (2050, 1152, 4608)])
def test_linear_bf16_residual_epilogues(M, N, K):
    say(f"linear bf16 residual {M}x{N}x{K}")
    A, W, b = rnd(4, (M, K)), rnd(5, (N, K), 0.05), rnd(6, (N,), 0.1)
    x0 = rnd(8, (M, N), bf=False)
    gate = rnd(9, (N,), 0.5, bf=False)
    ref = dit.linear(A.astype(np.float64), W.astype(np.float64), b.astype(np.float64))
    _, x, xc = run_linear(_lib.T2I_BF16, _lib.T2I_EPI_RESID, A, W, b, resid=x0, with_copy=True)
    xg = x.cpu().numpy()
    assert rel_l2(xg.astype(np.float64) - x0, ref) < 1e-4
    assert np.array_equal(xc.float().cpu().numpy(), synth.round_bf16(xg))
    _, x, _ = run_linear(_lib.T2I_BF16, _lib.T2I_EPI_RESID_GATED, A, W, b, resid=x0, gate=gate)
    assert rel_l2(x.cpu().numpy().astype(np.float64) - x0, gate * ref) < 1e-4


WIDE_SHAPES = [(4096, 12288, 3072, 1), (4096, 9216, 3072, 0), (4096, 3072, 3072, 4),
               (4096, 3072, 12288, 4), (3000, 3072, 3072, 0), (2048, 4096, 2048, 1)]


@pytest.mark.parametrize("M,N,K,epi", WIDE_SHAPES)
def test_linear_bf16_wide_sampled_rows(M, N, K, epi):
    """The 3072-wide model's projections (256x256 / 256x192 / 256x128 tiles,
    long K) on sampled rows."""
    say(f"linear bf16 wide {M}x{N}x{K} epi {epi}")
    A, W, b = rnd(60, (M, K)), rnd(61, (N, K), 0.03), rnd(62, (N,), 0.1)
    x0 = rnd(63, (M, N), bf=False) if epi >= 3 else None
    gate = rnd(64, (N,), 0.5, bf=False) if epi == 4 else None
    out, x, _ = run_linear(_lib.T2I_BF16, epi, A, W, b, resid=x0, gate=gate)
    rows = np.r_[np.arange(0, M, 97), M - 1]
    ref = dit.linear(A[rows].astype(np.float64), W.astype(np.float64), b.astype(np.float64))
    if epi == 0:
        got = to_host(out)[rows]
    elif epi == 1:
        got, ref = to_host(out)[rows], dit.gelu_tanh(ref)
    else:
        got, ref = x.cpu().numpy().astype(np.float64)[rows] - x0[rows], gate * ref
    err = rel_l2(got, ref)
    say(f"  rel_l2 {err:.2e}")
    assert err < (3e-3 if epi < 3 else 1e-4)


def test_linear_bf16_operand_over_2gib():
    """An A operand past 2^31 bytes (M = 2^20 + 37 rows of K = 1024): the
    direct-load tiles address operands with 32-bit offsets, so the library
    takes the register-staged tiles here; sampled rows, the last included,
    against the oracle."""
    lib = t2i.load()
    M, N, K = (1 << 20) + 37, 144, 1024
    assert 2 * M * K > 0x7fffffff
    g = torch.Generator(device=DEV).manual_seed(70)
    dA = torch.randn(M, K, generator=g, device=DEV).to(torch.bfloat16)
    W, b = rnd(71, (N, K), 0.05), rnd(72, (N,), 0.1)
    dW, db = to_dev(W, "bf16"), to_dev(b, "bf16")
    out = torch.zeros((M, N), dtype=torch.bfloat16, device=DEV)
    say("linear bf16 with a 2 GiB+ operand")
    _lib.check(lib.t2i_op_linear(_lib.T2I_BF16, 0, M, N, K, dA.data_ptr(), K, dW.data_ptr(), K,
                                 db.data_ptr(), out.data_ptr(), N, None, 0, None, None,
                                 _stream()))
    torch.cuda.synchronize()
    rows = [0, 1, 4097, 1 << 19, (1 << 20) - 1, M - 2, M - 1]
    A_rows = dA[rows].float().cpu().numpy().astype(np.float64)
    ref = dit.linear(A_rows, W.astype(np.float64), b.astype(np.float64))
    err = rel_l2(out[rows].float().cpu().numpy(), ref)
    say(f"  rel_l2 {err:.2e}")
    assert err < 3e-3
    del dA, out
    torch.cuda.empty_cache()


@pytest.mark.parametrize("M,N,K,epi", [(64, 128, 256, 0), (100, 520, 128, 2), (77, 33, 90, 4)])
def test_linear_f32(M, N, K, epi):
    A, W, b = rnd(10, (M, K), bf=False), rnd(11, (N, K), 0.05, bf=False), rnd(12, (N,), 0.1, bf=False)
    x0 = rnd(13, (M, N), bf=False)
    gate = rnd(14, (N,), 0.5, bf=False)
    ref = dit.linear(A.astype(np.float64), W.astype(np.float64), b.astype(np.float64))
    out, x, _ = run_linear(_lib.T2I_F32, epi, A, W, b, resid=x0 if epi >= 3 else None,
                           gate=gate if epi == 4 else None)
    if epi == 0:
        assert rel_l2(to_host(out), ref) < 1e-6
    elif epi == 2:
        assert rel_l2(to_host(out), dit.silu(ref)) < 1e-6
    else:
        assert rel_l2(x.cpu().numpy().astype(np.float64) - x0, gate * ref) < 1e-6


def run_attention(dtype, heads, d, seqs, q, k, v, seg2=None):
    """seqs: (q_start, q_len, k_start, k_len); seg2: (k2_start, k2_len) per sequence."""
    lib = t2i.load()
    n = len(seqs)
    qs, ql, ks, kl = ((C.c_int32 * n)(*[s[i] for s in seqs]) for i in range(4))
    k2s = k2l = None
    if seg2 is not None:
        k2s, k2l = ((C.c_int32 * n)(*[s[i] for s in seg2]) for i in range(2))
    dt = "bf16" if dtype == _lib.T2I_BF16 else "f32"
    w = heads * d
    if dtype == _lib.T2I_BF16:
        # bf16 kernels read V transposed, token stride padded to 64
        ldv = (v.shape[0] + 63) // 64 * 64
        vt = np.zeros((w, ldv), dtype=np.float32)
        vt[:, :v.shape[0]] = v.T
        vt[:, v.shape[0]:] = np.nan          # padding must never be read into results
        v_dev, ldv_arg = to_dev(vt, dt), ldv
    else:
        v_dev, ldv_arg = to_dev(v, dt), w
    dq, dk = to_dev(q, dt), to_dev(k, dt)
    o = torch.zeros(dq.shape, dtype=dq.dtype, device=DEV)
    st = lib.t2i_op_attention(dtype, heads, d, n, qs, ql, ks, kl, k2s, k2l, dq.data_ptr(), w,
                              dk.data_ptr(), w, v_dev.data_ptr(), ldv_arg, o.data_ptr(), w,
                              _stream())
    _lib.check(st)
    torch.cuda.synchronize()
    return to_host(o)


def run_cross_attention(heads, d, seqs, q, k, v):
    """seqs: (q_start, q_len, k_start, k_len); bf16, V passed transposed."""
    lib = t2i.load()
    n = len(seqs)
    qs, ql, ks, kl = ((C.c_int32 * n)(*[s[i] for s in seqs]) for i in range(4))
    w = heads * d
    ldv = (v.shape[0] + 63) // 64 * 64
    vt = np.zeros((w, ldv), dtype=np.float32)
    vt[:, :v.shape[0]] = v.T
    vt[:, v.shape[0]:] = np.nan              # padding must never be read into results
    dq, dk, dv = to_dev(q, "bf16"), to_dev(k, "bf16"), to_dev(vt, "bf16")
    o = torch.zeros(dq.shape, dtype=dq.dtype, device=DEV)
    st = lib.t2i_op_cross_attention(_lib.T2I_BF16, heads, d, n, qs, ql, ks, kl, dq.data_ptr(), w,
                                    dk.data_ptr(), w, dv.data_ptr(), ldv, o.data_ptr(), w,
                                    _stream())
    _lib.check(st)
    torch.cuda.synchronize()
    return to_host(o)


def _text_seqs(q_lens, k_lens):
    """Packed query sequences, each with its own text block starting at a multiple of 8."""
    seqs, q0, k0 = [], 0, 0
    for nq, nk in zip(q_lens, k_lens):
        seqs.append((q0, nq, k0, nk))
        q0 += nq
        k0 += (nk + 7) // 8 * 8
    return seqs, q0, k0


# (name, heads, query lengths, text lengths).  The two-tile kernel takes two
# 128-query tiles per workgroup from 1024 (tile, head) pairs on: the 1024-px
# guided shape (2 x 4096 queries, 16 heads, 120 keys); 21 sequences of three
# tiles each plus one of one tile (64 tiles), so that many workgroups take
# their two tiles from two sequences with different texts (ragged, 1 key, a
# full 128); a small launch of one tile per workgroup; a text longer than 128
# keys (the pipelined kernel).
CROSS_CASES = [
    ("guided-1024px", 16, [4096, 4096], [120, 120]),
    ("straddling-pairs", 16, [384] * 21 + [100], [120, 77, 1, 128, 64, 13, 8] * 3 + [50]),
    ("one-tile-per-group", 4, [500, 300], [120, 77]),
    ("long-text", 4, [300, 200], [200, 130]),
]


@pytest.mark.parametrize("name,H,q_lens,k_lens", CROSS_CASES, ids=[c[0] for c in CROSS_CASES])
def test_cross_attention_bf16(name, H, q_lens, k_lens):
    say(f"cross-attention bf16 {name}")
    d = 72
    seqs, nq, nk = _text_seqs(q_lens, k_lens)
    q, k, v = rnd(40, (nq, H * d)), rnd(41, (nk, H * d)), rnd(42, (nk, H * d))
    got = run_cross_attention(H, d, seqs, q, k, v)
    ref = attention_ref(seqs, q, k, v, H)
    err = rel_l2(got, ref)
    row_err = np.linalg.norm(got - ref, axis=1) / np.linalg.norm(ref, axis=1)
    say(f"  rel_l2 {err:.2e}, worst row {row_err.max():.2e}")
    assert err < 6e-3
    assert row_err.max() < 3e-2


def run_linear_cross_attention(fused, heads, d, seqs, A, W, b, k, v):
    """The query projection + cross-attention op (bf16, V passed transposed)."""
    lib = t2i.load()
    n = len(seqs)
    qs, ql, ks, kl = ((C.c_int32 * n)(*[s[i] for s in seqs]) for i in range(4))
    w = heads * d
    M, K = A.shape
    ldv = (v.shape[0] + 63) // 64 * 64
    vt = np.zeros((w, ldv), dtype=np.float32)
    vt[:, :v.shape[0]] = v.T
    vt[:, v.shape[0]:] = np.nan              # padding must never be read into results
    dA, dW, db = to_dev(A, "bf16"), to_dev(W, "bf16"), to_dev(b, "bf16")
    dk, dv = to_dev(k, "bf16"), to_dev(vt, "bf16")
    qbuf = None if fused else torch.zeros((M, w), dtype=torch.bfloat16, device=DEV)
    o = torch.zeros((M, w), dtype=torch.bfloat16, device=DEV)
    st = lib.t2i_op_linear_cross_attention(
        fused, heads, d, n, qs, ql, ks, kl, K, dA.data_ptr(), K, dW.data_ptr(), K, db.data_ptr(),
        dk.data_ptr(), w, dv.data_ptr(), ldv, qbuf.data_ptr() if qbuf is not None else None, w,
        o.data_ptr(), w, _stream())
    _lib.check(st)
    torch.cuda.synchronize()
    return o


# (name, heads, query lengths, text lengths, K): the 1024-px guided shape
# (16 heads, 2 x 4096 queries, 120 text keys, K = 1152); packed sequences of
# 256-row multiples with texts of 77 keys (a ragged last chunk), 1 key and a
# full 128; a narrow projection with K = 192 (one pass of the 3-stage ring)
# and one with K = 576
XQ_CASES = [
    ("guided-1024px", 16, [4096, 4096], [120, 120], 1152),
    ("packed-texts", 16, [256, 512, 1024, 256], [120, 77, 1, 128], 1152),
    ("narrow-k192", 4, [256, 768], [64, 8], 192),
    ("k576", 2, [512], [13], 576),
]


@pytest.mark.parametrize("name,H,q_lens,k_lens,K", XQ_CASES, ids=[c[0] for c in XQ_CASES])
def test_linear_cross_attention_fused_equals_two_launches(name, H, q_lens, k_lens, K):
    """The fused query projection + cross-attention kernel gives the bits of
    the projection and the cross-attention kernel run one after the other,
    and both match the oracle's projection and attention."""
    say(f"query projection + cross-attention {name}")
    d = 72
    seqs, nq, nk = _text_seqs(q_lens, k_lens)
    A, W, b = rnd(50, (nq, K)), rnd(51, (H * d, K), 0.05), rnd(52, (H * d,), 0.1)
    k, v = rnd(53, (nk, H * d)), rnd(54, (nk, H * d))
    fused = run_linear_cross_attention(1, H, d, seqs, A, W, b, k, v)
    two = run_linear_cross_attention(0, H, d, seqs, A, W, b, k, v)
    assert torch.equal(fused, two)
    q = dit.linear(A.astype(np.float64), W.astype(np.float64), b.astype(np.float64))
    ref = attention_ref(seqs, q, k, v, H)
    got = to_host(fused)
    err = rel_l2(got, ref)
    row_err = np.linalg.norm(got - ref, axis=1) / np.linalg.norm(ref, axis=1)
    say(f"  bitwise equal to two launches; rel_l2 {err:.2e}, worst row {row_err.max():.2e}")
    assert err < 6e-3
    assert row_err.max() < 3e-2


def attention_ref(seqs, q, k, v, heads):
    out = np.zeros(q.shape)
    for (q0, nq, k0, nk) in seqs:
        out[q0:q0 + nq] = dit.attention(q[q0:q0 + nq].astype(np.float64),
                                        k[k0:k0 + nk].astype(np.float64),
                                        v[k0:k0 + nk].astype(np.float64), heads)
    return out


ATTN_CASES = [
    ("self-ragged", 4, 72, [(0, 333, 0, 333)], 333, 333),
    ("varlen", 2, 72, [(0, 256, 0, 256), (256, 1024, 256, 1024), (1280, 77, 1280, 72)], 1357, 1357),
    ("cross-120", 4, 72, [(0, 500, 0, 120), (500, 300, 120, 120)], 800, 240),
    ("single-key", 2, 72, [(0, 130, 0, 1)], 130, 1),
    ("ragged-keys", 2, 72, [(0, 70, 0, 77), (70, 300, 80, 13)], 370, 93),
    ("d128", 3, 128, [(0, 200, 0, 260)], 200, 260),
    ("d64", 2, 64, [(0, 129, 0, 64)], 129, 64),
]


@pytest.mark.parametrize("name,H,d,seqs,nq,nk", ATTN_CASES, ids=[c[0] for c in ATTN_CASES])
def test_attention_bf16(name, H, d, seqs, nq, nk):
    say(f"attention bf16 {name}")
    q, k, v = rnd(20, (nq, H * d)), rnd(21, (nk, H * d)), rnd(22, (nk, H * d))
    got = run_attention(_lib.T2I_BF16, H, d, seqs, q, k, v)
    ref = attention_ref(seqs, q, k, v, H)
    err = rel_l2(got, ref)
    say(f"  rel_l2 {err:.2e}")
    assert err < 6e-3


def test_attention_bf16_identical_keys_give_mean():
    H, d, n = 2, 72, 300
    q = rnd(23, (n, H * d))
    k = np.tile(rnd(24, (1, H * d)), (n, 1))
    v = rnd(25, (n, H * d))
    got = run_attention(_lib.T2I_BF16, H, d, [(0, n, 0, n)], q, k, v)
    ref = np.tile(v.astype(np.float64).mean(axis=0), (n, 1))
    assert rel_l2(got, ref) < 6e-3


def test_attention_bf16_full_size_sampled_rows():
    """1024 px self-attention: 2 sequences x 4096 tokens, 16 heads of 72."""
    H, d, n = 16, 72, 4096
    q, k, v = rnd(26, (2 * n, H * d)), rnd(27, (2 * n, H * d)), rnd(28, (2 * n, H * d))
    seqs = [(0, n, 0, n), (n, n, n, n)]
    got = run_attention(_lib.T2I_BF16, H, d, seqs, q, k, v)
    rows = np.r_[np.arange(0, 2 * n, 97), n - 1, 2 * n - 1]
    ref = np.zeros((len(rows), H * d))
    for i, r in enumerate(rows):
        s0 = 0 if r < n else n
        ref[i] = dit.attention(q[r:r + 1].astype(np.float64), k[s0:s0 + n].astype(np.float64),
                               v[s0:s0 + n].astype(np.float64), H)[0]
    assert rel_l2(got[rows], ref) < 6e-3


@pytest.mark.parametrize("sharp", [4.0, 8.0, 16.0])
def test_attention_bf16_sharp_logits(sharp):
    """Large logits: queries scaled by 4..16 and key norms growing along the
    sequence, so that later key tiles keep raising the row maximum (the
    kernel's lazy rescale, taken when a score exceeds the kept maximum by 2^8,
    fires after the first tile) and the softmax is sharp."""
    H, d, nq, nk = 4, 72, 300, 1000
    q = synth.round_bf16(rnd(80, (nq, H * d)) * sharp)
    ramp = np.linspace(0.4, 1.6, nk, dtype=np.float32)[:, None]
    k = synth.round_bf16(rnd(81, (nk, H * d)) * ramp)
    v = rnd(82, (nk, H * d))
    seqs = [(0, nq, 0, nk)]
    got = run_attention(_lib.T2I_BF16, H, d, seqs, q, k, v)
    ref = attention_ref(seqs, q, k, v, H)
    err = rel_l2(got, ref)
    rows = np.linalg.norm(got - ref, axis=1) / np.linalg.norm(ref, axis=1)
    lg = np.abs(q[:, :d].astype(np.float64) @ k[:, :d].astype(np.float64).T) / np.sqrt(d)
    say(f"attention bf16 sharp x{sharp}: max |logit| {lg.max():.1f}, rel_l2 {err:.2e}, "
        f"worst row {rows.max():.2e}")
    assert err < 6e-3 and rows.max() < 3e-2


def _packed_keys(lengths):
    """Key row starts (multiples of 8, as the bf16 kernel requires) for
    sequences of the given key counts, and the total row count."""
    starts, at = [], 0
    for n in lengths:
        starts.append(at)
        at += (n + 7) // 8 * 8
    return starts, max(at, 8)


@pytest.mark.parametrize("d", [72, 128])
def test_attention_bf16_eight_wave_pipeline_edges(d):
    """16 heads x 16 sequences of 256 queries: 256 workgroups, so the 8-wave
    kernel runs (5-stage ring with one barrier per two key tiles at d = 72,
    4 stages at 128).  Key counts give 1 .. 8 key tiles, odd and even, full
    and ragged; a second call splits every sequence's keys into two ragged
    segments (the first segment's last tile ragged in the middle of the
    sequence)."""
    H, nq1 = 16, 256
    lens = [1, 63, 64, 65, 128, 130, 192, 200, 256, 300, 320, 333, 384, 400, 448, 460]
    starts, nk = _packed_keys(lens)
    q = rnd(60 + d, (16 * nq1, H * d))
    k, v = rnd(61 + d, (nk, H * d)), rnd(62 + d, (nk, H * d))
    seqs = [(i * nq1, nq1, starts[i], lens[i]) for i in range(16)]
    say(f"attention bf16 8-wave edges d={d}")
    got = run_attention(_lib.T2I_BF16, H, d, seqs, q, k, v)
    err = rel_l2(got, attention_ref(seqs, q, k, v, H))
    say(f"  one segment rel_l2 {err:.2e}")
    assert err < 6e-3
    # two segments: n1 + n2 keys, n1 ragged
    n1 = [1, 7, 40, 63, 65, 77, 100, 129, 1, 33, 64, 70, 130, 191, 200, 250]
    n2 = [64, 1, 100, 63, 65, 200, 13, 129, 300, 64, 1, 256, 70, 8, 192, 210]
    st1, tot1 = _packed_keys(n1)
    st2, tot2 = _packed_keys(n2)
    k = rnd(63 + d, (tot1 + tot2, H * d))
    v = rnd(64 + d, (tot1 + tot2, H * d))
    seqs = [(i * nq1, nq1, st1[i], n1[i]) for i in range(16)]
    seg2 = [(tot1 + st2[i], n2[i]) for i in range(16)]
    got = run_attention(_lib.T2I_BF16, H, d, seqs, q, k, v, seg2)
    ref = np.zeros(q.shape)
    for (q0, n_q, k0, n_k), (k20, n_k2) in zip(seqs, seg2):
        idx = np.r_[np.arange(k0, k0 + n_k), np.arange(k20, k20 + n_k2)]
        ref[q0:q0 + n_q] = dit.attention(q[q0:q0 + n_q].astype(np.float64),
                                         k[idx].astype(np.float64), v[idx].astype(np.float64), H)
    err = rel_l2(got, ref)
    say(f"  two segments rel_l2 {err:.2e}")
    assert err < 6e-3


@pytest.mark.parametrize("d", [64, 72])
def test_attention_bf16_packed_sequences_equal_each_alone(d):
    """16 heads, 11 sequences packed into one launch of 512 eight-wave
    workgroups.  Query counts give odd and even tile counts and ragged query
    tails (one query in a last tile); key counts run from 1 to 460 (ragged,
    single tile, several tiles); a second call splits the keys into two
    segments.  A sequence run on its own (a launch of two-wave workgroups,
    too few tiles to fill the chip with eight) gives the same bits, since a
    query's arithmetic does not depend on the workgroup size or on the other
    sequences of the launch."""
    H = 16
    q_lens = [600, 513, 1024, 256, 300, 777, 512, 1000, 260, 900, 520]
    k_lens = [1, 63, 130, 200, 64, 333, 460, 65, 8, 129, 256]
    q_starts = np.cumsum([0] + q_lens[:-1]).tolist()
    nq = sum(q_lens)
    starts, nk = _packed_keys(k_lens)
    q = rnd(70 + d, (nq, H * d))
    k, v = rnd(71 + d, (nk, H * d)), rnd(72 + d, (nk, H * d))
    seqs = [(q_starts[i], q_lens[i], starts[i], k_lens[i]) for i in range(len(q_lens))]
    say(f"attention bf16 packed sequences d={d}")
    got = run_attention(_lib.T2I_BF16, H, d, seqs, q, k, v)
    err = rel_l2(got, attention_ref(seqs, q, k, v, H))
    say(f"  one segment rel_l2 {err:.2e}")
    assert err < 6e-3
    for i in (0, 1, 5, 9):
        q0, n_q, k0, n_k = seqs[i]
        alone = run_attention(_lib.T2I_BF16, H, d, [(0, n_q, k0, n_k)], q[q0:q0 + n_q], k, v)
        assert np.array_equal(alone, got[q0:q0 + n_q]), i
    n1 = [1, 40, 65, 100, 129, 7, 200, 64, 33, 250, 8]
    n2 = [64, 100, 1, 13, 129, 300, 70, 192, 1, 210, 56]
    st1, tot1 = _packed_keys(n1)
    st2, tot2 = _packed_keys(n2)
    k = rnd(73 + d, (tot1 + tot2, H * d))
    v = rnd(74 + d, (tot1 + tot2, H * d))
    seqs = [(q_starts[i], q_lens[i], st1[i], n1[i]) for i in range(len(q_lens))]
    seg2 = [(tot1 + st2[i], n2[i]) for i in range(len(q_lens))]
    got = run_attention(_lib.T2I_BF16, H, d, seqs, q, k, v, seg2)
    ref = np.zeros(q.shape)
    for (q0, n_q, k0, n_k), (k20, n_k2) in zip(seqs, seg2):
        idx = np.r_[np.arange(k0, k0 + n_k), np.arange(k20, k20 + n_k2)]
        ref[q0:q0 + n_q] = dit.attention(q[q0:q0 + n_q].astype(np.float64),
                                         k[idx].astype(np.float64), v[idx].astype(np.float64), H)
    err = rel_l2(got, ref)
    say(f"  two segments rel_l2 {err:.2e}")
    assert err < 6e-3


JOINT_CASES = [
    # (name, H, d, [(q_start, q_len, k_start, k_len)], [(k2_start, k2_len)], nq, nk)
    ("txt+img", 2, 128, [(0, 64, 0, 64), (64, 256, 0, 64)], [(64, 256), (64, 256)], 320, 320),
    ("ragged-two-seqs", 3, 128, [(0, 77, 0, 40), (77, 130, 48, 23)],
     [(80, 130), (216, 77)], 207, 296),
    ("second-only", 2, 72, [(0, 100, 0, 0)], [(8, 93)], 100, 101),
    ("first-only", 2, 64, [(0, 70, 16, 50)], [(0, 0)], 70, 66),
]


@pytest.mark.parametrize("name,H,d,seqs,seg2,nq,nk", JOINT_CASES, ids=[c[0] for c in JOINT_CASES])
@pytest.mark.parametrize("dtype", [_lib.T2I_BF16, _lib.T2I_F32], ids=["bf16", "f32"])
def test_attention_two_key_segments(dtype, name, H, d, seqs, seg2, nq, nk):
    """Keys of a sequence in two separate row ranges == attention over their concatenation."""
    say(f"attention two segments {name} dtype {dtype}")
    bf = dtype == _lib.T2I_BF16
    q, k, v = rnd(50, (nq, H * d), bf=bf), rnd(51, (nk, H * d), bf=bf), rnd(52, (nk, H * d), bf=bf)
    got = run_attention(dtype, H, d, seqs, q, k, v, seg2)
    ref = np.zeros(q.shape)
    for (q0, n_q, k0, n_k), (k20, n_k2) in zip(seqs, seg2):
        idx = np.r_[np.arange(k0, k0 + n_k), np.arange(k20, k20 + n_k2)]
        ref[q0:q0 + n_q] = dit.attention(q[q0:q0 + n_q].astype(np.float64),
                                         k[idx].astype(np.float64), v[idx].astype(np.float64), H)
    err = rel_l2(got, ref)
    say(f"  rel_l2 {err:.2e}")
    assert err < (6e-3 if bf else 1e-6)


@pytest.mark.parametrize("H,d,seqs,nq,nk", [(2, 64, [(0, 64, 0, 64)], 64, 64),
                                            (2, 64, [(0, 64, 0, 16), (64, 10, 16, 16)], 74, 32)])
def test_attention_f32(H, d, seqs, nq, nk):
    q, k, v = (rnd(s, (n, H * d), bf=False) for s, n in ((30, nq), (31, nk), (32, nk)))
    got = run_attention(_lib.T2I_F32, H, d, seqs, q, k, v)
    assert rel_l2(got, attention_ref(seqs, q, k, v, H)) < 1e-6


@pytest.mark.parametrize("dtype,rows,D", [(1, 1000, 1152), (0, 64, 128), (1, 7, 3072)])
def test_ln_modulate(dtype, rows, D):
    lib = t2i.load()
    x = rnd(40, (rows, D), bf=False) * 2 + 0.5
    mod = rnd(41, (2, D), 0.3, bf=False)
    dx = torch.from_numpy(x.astype(np.float32)).to(DEV)
    dm = torch.from_numpy(mod.astype(np.float32)).to(DEV)
    out = torch.zeros((rows, D), dtype=torch.bfloat16 if dtype == 1 else torch.float32, device=DEV)
    _lib.check(lib.t2i_op_ln_modulate(dtype, rows, D, dx.data_ptr(), dm.data_ptr(),
                                      dm.data_ptr() + 4 * D, 1e-6, out.data_ptr(), _stream()))
    torch.cuda.synchronize()
    ref = dit.modulate(dit.layer_norm(x.astype(np.float64), 1e-6), mod[0], mod[1])
    assert rel_l2(to_host(out), ref) < (3e-3 if dtype == 1 else 1e-6)


def test_ln_modulate_bf16_row_count_does_not_change_bits():
    """Width 1152, bf16: launches of 1 .. 4104 rows (two rows per wave, odd
    counts leaving a wave one row) give the same bits on the same rows: a
    row's result does not depend on the batch; the rows match the oracle."""
    lib = t2i.load()
    D, rows = 1152, 4104
    x = rnd(42, (rows, D), bf=False) * 2 + 0.5
    mod = rnd(43, (2, D), 0.3, bf=False)
    dx = torch.from_numpy(x.astype(np.float32)).to(DEV)
    dm = torch.from_numpy(mod.astype(np.float32)).to(DEV)

    def run(n):
        out = torch.zeros((n, D), dtype=torch.bfloat16, device=DEV)
        _lib.check(lib.t2i_op_ln_modulate(1, n, D, dx.data_ptr(), dm.data_ptr(),
                                          dm.data_ptr() + 4 * D, 1e-6, out.data_ptr(), _stream()))
        torch.cuda.synchronize()
        return out

    big = run(rows)
    for n in (1, 255, 1024, 4095):
        assert torch.equal(run(n), big[:n]), n
    ref = dit.modulate(dit.layer_norm(x.astype(np.float64), 1e-6), mod[0], mod[1])
    assert rel_l2(to_host(big), ref) < 3e-3


@pytest.mark.parametrize("dtype,n_out,n_in,rank", [(1, 3072, 3072, 64), (1, 1152, 4608, 16),
                                                    (1, 1000, 1160, 40), (1, 77, 304, 128),
                                                    (1, 77, 300, 128), (0, 200, 130, 8)])
def test_lora_merge(dtype, n_out, n_in, rank):
    """W + alpha B A against the oracle: fp32 to 1e-6; bf16 equal to the oracle
    rounded to bf16 except where the fp32 sum lands on the other side of a
    rounding boundary (at most one bf16 step, on a tiny fraction)."""
    bf = dtype == 1
    W = rnd(70, (n_out, n_in), 0.05, bf=bf)
    A = rnd(71, (rank, n_in), 0.05, bf=bf)
    B = rnd(72, (n_out, rank), 0.05, bf=bf)
    alpha = 0.8
    dt = "bf16" if bf else "f32"
    dW, dA, dB = to_dev(W, dt), to_dev(A, dt), to_dev(B, dt)
    t2i.lora_merge(dW, dA, dB, alpha)
    torch.cuda.synchronize()
    from oracle import lora
    ref = lora.merge(W, A, B, alpha)
    got = to_host(dW)
    if not bf:
        assert rel_l2(got, ref) < 1e-6
        return
    ref_b = synth.round_bf16(ref.astype(np.float32)).astype(np.float64)
    diff = got != ref_b
    frac = diff.mean()
    say(f"lora {n_out}x{n_in} r{rank}: {frac:.2e} of elements one rounding step off")
    assert frac < 1e-3
    # a mismatch is one bf16 step of the larger of the two values (plus fp32
    # accumulation slack where W and alpha B A nearly cancel)
    d = np.abs(got[diff] - ref[diff])
    assert np.all(d <= np.maximum(np.abs(ref[diff]), np.abs(got[diff])) * 2.0 ** -7 + 1e-6)


def test_dma_read_calibration_kernel():
    """The counter-calibration read through the direct-to-LDS path runs and
    lands the source's bytes in LDS (every workgroup reports a 1.0 it read)."""
    lib = t2i.load()
    a = torch.ones(1 << 20, dtype=torch.float32, device=DEV)      # 4 MiB
    sink = torch.zeros(1024, dtype=torch.float32, device=DEV)
    _lib.check(lib.t2i_op_dma_read(C.c_void_p(a.data_ptr()), 4 << 20, C.c_void_p(sink.data_ptr()),
                                   _stream()))
    torch.cuda.synchronize()
    assert torch.all(sink == 1.0)
    assert lib.t2i_op_dma_read(C.c_void_p(a.data_ptr()), 1000, C.c_void_p(sink.data_ptr()),
                               _stream()) == 2


@pytest.mark.parametrize("dtype,n_out,n_in,rank", [(1, 300, 256, 24), (1, 64, 1160, 128),
                                                    (0, 70, 130, 8), (1, 77, 300, 16)])
def test_lora_merge_batch_equals_single_merges(dtype, n_out, n_in, rank):
    """One launch over several weights of a shape == one merge per weight, bitwise."""
    bf = dtype == 1
    dt = "bf16" if bf else "f32"
    n = 3
    Ws = [rnd(90 + i, (n_out, n_in), 0.05, bf=bf) for i in range(n)]
    As = [rnd(95 + i, (rank, n_in), 0.05, bf=bf) for i in range(n)]
    Bs = [rnd(99 + i, (n_out, rank), 0.05, bf=bf) for i in range(n)]
    one = [to_dev(w, dt) for w in Ws]
    bat = [to_dev(w, dt) for w in Ws]
    dA = [to_dev(a, dt) for a in As]
    dB = [to_dev(b, dt) for b in Bs]
    for w, a, b in zip(one, dA, dB):
        t2i.lora_merge(w, a, b, 0.7)
    t2i.lora_merge_batch(bat, dA, dB, 0.7)
    torch.cuda.synchronize()
    for x, y in zip(one, bat):
        assert torch.equal(x, y)
