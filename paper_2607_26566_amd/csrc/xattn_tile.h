// Cross-attention of image queries to a short text (at most 128 keys, two
// 64-key tiles), the pieces shared by the standalone kernel
// (attn_cross_kernel, attention.hip) and the query projection that ends in
// it (gemm_dma_kernel with XAttnArgs, gemm_dma.hip).  Both use these
// functions for the same arithmetic, so a query's output does not depend on
// which kernel computed it.
//
// LDS layouts of one head's text tile (64 keys):
//   * K: 64 rows of head_dim bf16, row r holding key swap23(r) of the tile
//     (chunk slots swizzled for pitches that are multiples of 64 bytes);
//   * V^T: row d (0 .. head_dim-1) = 64 keys in natural order, 16-byte chunk
//     c in slot c ^ ((d >> 1) & 7), then a row of ones (row head_dim) whose
//     products are the row sums of the probabilities.  The P V MFMAs also
//     read rows head_dim+1 .. 32*ceil(head_dim/32)-1 from whatever follows;
//     they only feed output rows that are never used.
#pragma once

#include "t2i_internal.h"

namespace t2i {

// Key order inside a staged K tile.  The P V MFMA's B operand is the lane's
// own probabilities: for 16-key chunk q a lane of half h holds S^T rows
// 16q + 8a + 4h + j (a in 0..1, j in 0..3), which the MFMA consumes as k-index
// 8h + 4a + j.  Staging key swap23(r) in K row r (bits 2 and 3 swapped) makes
// that k-index the natural key order, so V^T tiles stay in key order and can
// be copied to LDS unchanged.
__device__ __forceinline__ int swap23(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

template <int HD>
struct XTile {
  static constexpr int BKV = 64;
  static constexpr int DC = (HD + 15) / 16;   // 16-wide d chunks of S^T = K Q^T
  static constexpr int DT = (HD + 31) / 32, HDO = DT * 32;
  static constexpr bool ONES = HD < HDO;      // row sums from the ones row of V^T
  static constexpr int CPR = HD / 8, PK = 2 * HD, NI = 2 * CPR;   // NI: DMA instructions per tile
  static constexpr int KRS = (CPR == 4 || CPR == 8 || CPR == 16) ? 16 / CPR : 0;
  static constexpr int VROWS = ONES ? HD + 1 : HDO;   // V^T rows kept
  static constexpr int KSTAGE = BKV * PK, VSTAGE = VROWS * 128;
  static_assert(HD % 8 == 0 && KSTAGE % 1024 == 0, "head dim");
};

// DMA instruction i (0 .. NI-1) of head hh's text tile starting at key kv0
// (the text ends at k_end): instructions 0 .. CPR-1 fill the K tile at kdst,
// the rest the V^T rows at vdst; 1 KB each, 16 bytes per lane.  Keys past
// the text are clamped to its last key (their scores are masked); V^T chunks
// wholly past it are read from the tile's first chunk (their probabilities
// are 0).  Byte offsets stay below 2^31 (the launchers check).
template <int HD>
__device__ __forceinline__ void xattn_dma(__amdgpu_buffer_rsrc_t rk, __amdgpu_buffer_rsrc_t rv, int i,
                                          int kv0, int k_end, int hh, int ldk, int ldvt, char* kdst,
                                          char* vdst) {
  using X = XTile<HD>;
  const int lane = threadIdx.x & 63;
  if (i < X::CPR) {
    const int o = i * 1024 + lane * 16, r = o / X::PK, slot = (o - r * X::PK) / 16;
    const int c = X::KRS ? slot ^ ((r / X::KRS) & (X::CPR - 1)) : slot;
    const int key = min(kv0 + swap23(r), k_end - 1);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rk, (__attribute__((address_space(3))) void*)(kdst + i * 1024), 16,
        2u * (uint32_t)(key * ldk + hh * HD + c * 8), 0, 0, 0);
  } else {
    const int o = (i - X::CPR) * 1024 + lane * 16, d = o / 128;
    const int gk = kv0 + 8 * ((lane & 7) ^ ((d >> 1) & 7));
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rv, (__attribute__((address_space(3))) void*)(vdst + (i - X::CPR) * 1024), 16,
        2u * (uint32_t)((hh * HD + d) * ldvt + (gk < k_end ? gk : kv0)), 0, 0, 0);
  }
}

// The ones row of a V^T tile (the DMA never writes it); threads tid0 .. of a
// workgroup of nthreads write its 64 entries
template <int HD>
__device__ __forceinline__ void xattn_ones(char* vt, int tid, int nthreads) {
  if constexpr (XTile<HD>::ONES)
    for (int i = tid; i < 64; i += nthreads) ((bf16*)(vt + HD * 128))[i] = (bf16)1.f;
}

// After the tile loads of a text of nkeys keys have landed in the last tile's
// V^T at vt: a chunk the text ends inside holds bytes from beyond it; zero
// the columns past the text (their probabilities are 0).  The caller
// synchronises afterwards when this returns true.
template <int HD>
__device__ __forceinline__ bool xattn_fix_ragged(char* vt, int nkeys, int tid, int nthreads) {
  if (!(nkeys & 7)) return false;
  const int c0 = nkeys - ((nkeys - 1) / 64) * 64;   // valid columns of the last tile
  for (int i = tid; i < HD * 64; i += nthreads) {
    const int d = i >> 6, col = i & 63;
    if (col >= c0)
      *(bf16*)(vt + d * 128 + (((col >> 3) ^ ((d >> 1) & 7)) << 4) + (col & 7) * 2) = (bf16)0.f;
  }
  return true;
}

// One wave's 32 queries (lane: query ql = lane & 31, d half hl = lane >> 5)
// against the nkeys (1 .. 128) keys of one head held in LDS tiles k0 / v0
// (keys 0 .. 63) and k1 / v1 (64 .. 127).  qf: the query's fragments as
// the B operand of S^T = K Q^T (d = 16c + 8hl .. +7, zero past HD).  All
// scores are computed first and the softmax takes the exact row maximum;
// probabilities exp2(sc (s - max)), sc = 1 for a pre-scaled Q (QS), else
// scale_log2.  Lanes whose query lies inside the sequence (valid) hand
// their output, four consecutive values d .. d+3 at a time, to out(d, w).
template <int HD, bool QS, class Out>
__device__ __forceinline__ void xattn_wave(const char* k0, const char* k1, const char* v0,
                                           const char* v1, int nkeys,
                                           const bf16x8 (&qf)[XTile<HD>::DC], float scale_log2,
                                           bool valid, Out&& out) {
  using X = XTile<HD>;
  constexpr int DC = X::DC, DT = X::DT, CPR = X::CPR, PK = X::PK, KRS = X::KRS;
  const int lane = threadIdx.x & 63, ql = lane & 31, hl = lane >> 5;
  const int nt = (nkeys + X::BKV - 1) / X::BKV;
  auto kst = [&](int t) { return t == 0 ? k0 : k1; };
  auto vst = [&](int t) { return t == 0 ? v0 : v1; };

  // S^T of both tiles (the first MFMA of each sum takes a zero accumulator)
  f32x16 sc_[2][2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    if (t >= nt) break;
#pragma unroll
    for (int c = 0; c < DC; ++c) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const int rr = 32 * kb + ql, cc = 2 * c + hl;
        bf16x8 kf = bf16x8{};
        if (cc < CPR) {
          const int slot = KRS ? cc ^ ((rr / KRS) & (CPR - 1)) : cc;
          kf = *(const bf16x8*)(kst(t) + rr * PK + slot * 16);
        }
        sc_[t][kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[c],
                                                             c == 0 ? f32x16{} : sc_[t][kb], 0, 0, 0);
      }
    }
  }
  // Element e of key block kb is key swap23(32 kb + 8 (e >> 2) + (e & 3)) + 8 hl
  // of its tile (swap23 moves the lane-half bit 2 to bit 3): only the ragged
  // last tile is masked, against a per-lane threshold and compile-time offsets
  float mx = -INFINITY;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    if (t >= nt) break;
    const int valid = nkeys - t * X::BKV;
    if (valid < X::BKV) {
      const int thr = valid - 8 * hl;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (swap23(32 * kb + 8 * (e >> 2) + (e & 3)) >= thr) sc_[t][kb][e] = -INFINITY;
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sc_[t][kb][e]);
  }
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));   // the query's keys sit in lanes ql and ql + 32
  // probabilities exp2(sc * (s - mx)): a subtraction, or one fma per score
  const float sc = QS ? 1.0f : scale_log2;
  const float mxs = mx * sc;

  // P V over both tiles; row sums from the ones row or per lane
  f32x16 o[DT];
  float psum = 0.f;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    if (t >= nt) break;
    const char* vb = vst(t);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      bf16x8 pf;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = sc_[t][q >> 1][8 * (q & 1) + e];
        const float p = __builtin_amdgcn_exp2f(QS ? x - mx : fmaf(x, sc, -mxs));
        if (!X::ONES) psum += p;
        pf[e] = (bf16)p;
      }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int row = dt * 32 + ql;
        const bf16x8 vf =
            *(const bf16x8*)(vb + row * 128 + (((2 * q + hl) ^ ((row >> 1) & 7)) << 4));
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, t == 0 && q == 0 ? f32x16{} : o[dt],
                                                        0, 0, 0);
      }
    }
  }
  float l;
  if (X::ONES) {
    constexpr int RR = HD % 32;
    l = __shfl(o[HD / 32][4 * (RR / 8) + (RR % 4)], ((RR % 8) / 4) * 32 + ql, 64);
  } else {
    l = psum + __shfl_xor(psum, 32, 64);
  }
  if (valid) {
    const float inv = 1.0f / l;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d = dt * 32 + i * 8 + hl * 4;
        if (d < HD) {
          bf16x4 w;
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) w[jj] = (bf16)(o[dt][4 * i + jj] * inv);
          out(d, w);
        }
      }
  }
}

}  // namespace t2i
