// Linear layers y = A W^T + b of the DiT block (qkv, out, cross-q, cross-out,
// fc1, fc2, text projections) on gfx950.
//
//  * gemm_bf16_kernel: bf16 operands, fp32 accumulation on MFMA
//    (v_mfma_f32_16x16x32_bf16).  A workgroup of 4 waves owns a BM x BN output
//    tile; each wave a (BM/2) x (BN/2) quadrant.  K advances 64 at a time
//    through double-buffered LDS tiles (row pitch 72 bf16 = 144 B, so the 16
//    rows a fragment load touches fall in distinct bank groups); the next K
//    tile is fetched from HBM into registers while MFMA works on the current
//    one.  Workgroups are numbered so that each XCD (dispatched round-robin)
//    receives a contiguous run of output tiles: tiles sharing A rows share
//    that XCD's L2.
//  * gemm_f32_kernel: SIMT fp32 FMA for the fp32 model's layers.
//  * linear_rows_kernel: the conditioning GEMMs (timestep MLP, adaLN table),
//    8 timesteps per pass, weight-streaming and HBM-bound; its per-element
//    summation order does not depend on the number of timesteps, so a
//    sample's batched table equals the per-step tables bitwise.
//
// Epilogues (bias always added): store, GELU-tanh, SiLU, residual add,
// gated residual add (gate row chosen by the row's sequence), and split-store
// for fused q|k|v projections: q and k row-major, v transposed (V^T[d][token],
// four tokens per 8-byte store) so attention can stage V^T tiles directly.
#include <algorithm>
#include <cstring>

#include "t2i_internal.h"

namespace t2i {

hipError_t launch_gemm_dma(const bf16* A, int lda, const bf16* W, int ldw, const bf16* bias,
                           int M, int N, int K, int kind, const Epi& epi, int vec_ok,
                           hipStream_t st);
hipError_t launch_gemm_dma_small(const bf16* A, int lda, const bf16* W, int ldw, const bf16* bias,
                                 int M, int N, int K, int kind, const Epi& epi, int vec_ok,
                                 hipStream_t st);

// Map launch order -> tile order so XCD x (blocks b with b % 8 == x) owns the
// contiguous tile range of its share.
__device__ __forceinline__ int xcd_remap(int b, int nb) {
  const int q = nb >> 3, r = nb & 7;
  const int x = b & 7, j = b >> 3;
  return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + j;
}

// Epilogue on four consecutive columns nb..nb+3 of row m (vector path).
template <int KIND>
__device__ __forceinline__ void epi_store4(const Epi& e, int m, int nb, const float v[4]) {
  if (KIND == EPI_STORE_F32) {
    *(float4*)((float*)e.out + (size_t)m * e.ldo + nb) = float4{v[0], v[1], v[2], v[3]};
  } else if (KIND == EPI_STORE || KIND == EPI_GELU || KIND == EPI_SILU) {
    bf16x4 w;
    const float qs = KIND == EPI_STORE && nb < e.qcols ? e.qscale : 1.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float y = v[r];
      if (KIND == EPI_GELU) y = gelu_tanh(y);
      if (KIND == EPI_SILU) y = silu(y);
      if (KIND == EPI_STORE) y *= qs;
      w[r] = (bf16)y;
    }
    *(bf16x4*)((bf16*)e.out + (size_t)m * e.ldo + nb) = w;
  } else {
    float4 g4 = float4{1.f, 1.f, 1.f, 1.f};
    if (KIND == EPI_RESID_GATED)
      g4 = *(const float4*)(e.gate + (size_t)e.map.modrow[seq_of_row(e.map, m)] * e.ld_gate + nb);
    float4* xp = (float4*)(e.x + (size_t)m * e.ldx + nb);
    float4 x4 = *xp;
    x4.x += g4.x * v[0];
    x4.y += g4.y * v[1];
    x4.z += g4.z * v[2];
    x4.w += g4.w * v[3];
    *xp = x4;
    if (e.xb) {
      bf16x4 w{(bf16)x4.x, (bf16)x4.y, (bf16)x4.z, (bf16)x4.w};
      *(bf16x4*)(e.xb + (size_t)m * e.ldx + nb) = w;
    }
  }
}

// BM x BN tile per workgroup of 4 waves arranged WGM x (4 / WGM).  Except for
// the split q|k|v store, the MFMA computes C^T fragments (operands swapped),
// so a lane ends with four consecutive output columns of one row and the
// epilogue issues one 8-byte (bf16) or 16-byte (fp32) access per lane.
template <int BM, int BN, int WGM, int KIND>
__device__ __forceinline__ void gemm_bf16_body(const bf16* __restrict__ A, int lda,
                                               const bf16* __restrict__ W, int ldw,
                                               const bf16* __restrict__ bias, int M, int N, int K,
                                               const Epi& epi, int tiles_n, int vec_ok, int tile) {
  constexpr bool PART = KIND == EPI_PARTIAL;
  constexpr int EK = PART ? EPI_STORE_F32 : KIND;
  constexpr int BK = 64;
  constexpr int LDK = BK + 8;
  constexpr int WGN = 4 / WGM;
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int ACH = BM * (BK / 8), BCH = BN * (BK / 8);   // 16-byte chunks per tile
  constexpr int APT = (ACH + 255) / 256, BPT = (BCH + 255) / 256;
  constexpr bool CT = KIND != EPI_SPLIT_VT;
  static_assert(WM % 16 == 0 && WN % 16 == 0, "wave tile");
  __shared__ bf16 As[2][BM * LDK];
  __shared__ bf16 Bs[2][BN * LDK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int m0 = (tile / tiles_n) * BM, n0 = (tile % tiles_n) * BN;

  const bf16* Ap[APT];
  const bf16* Bp[BPT];
#pragma unroll
  for (int i = 0; i < APT; ++i) {
    const int c = min(tid + 256 * i, ACH - 1);
    Ap[i] = A + (size_t)min(m0 + (c >> 3), M - 1) * lda + (c & 7) * 8;
  }
#pragma unroll
  for (int i = 0; i < BPT; ++i) {
    const int c = min(tid + 256 * i, BCH - 1);
    Bp[i] = W + (size_t)min(n0 + (c >> 3), N - 1) * ldw + (c & 7) * 8;
  }

  bf16x8 ra[APT], rb[BPT];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < APT; ++i)
      if (ACH % 256 == 0 || tid + 256 * i < ACH) ra[i] = *(const bf16x8*)(Ap[i] + k0);
#pragma unroll
    for (int i = 0; i < BPT; ++i)
      if (BCH % 256 == 0 || tid + 256 * i < BCH) rb[i] = *(const bf16x8*)(Bp[i] + k0);
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < APT; ++i) {
      const int c = tid + 256 * i;
      if (ACH % 256 == 0 || c < ACH) *(bf16x8*)&As[buf][(c >> 3) * LDK + (c & 7) * 8] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
      const int c = tid + 256 * i;
      if (BCH % 256 == 0 || c < BCH) *(bf16x8*)&Bs[buf][(c >> 3) * LDK + (c & 7) * 8] = rb[i];
    }
  };

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Epilogue operands of a tile that is whole in N (as in gemm_dma.hip): the
  // BN bias values and, for a gated update whose rows all belong to one
  // sequence, the BN gate values, fetched with the first tile and kept in LDS,
  // so that the epilogue's stores never wait behind a global load.
  constexpr bool GATED = KIND == EPI_RESID_GATED;
  __shared__ __attribute__((aligned(16))) float ebias[BN];
  __shared__ __attribute__((aligned(16))) float egate[GATED ? BN : 4];
  const bool whole_n = !PART && vec_ok && n0 + BN <= N;
  bool one_seq = false;
  int grow = 0;
  if constexpr (GATED) {
    const int s0 = seq_of_row(epi.map, m0), s1 = seq_of_row(epi.map, min(m0 + BM, M) - 1);
    one_seq = whole_n && s0 == s1;
    grow = epi.map.modrow[s0];
  }
  const bool stager = tid < BN / 4;
  bf16x4 sbias{};
  float4 sgate{};
  if (whole_n && stager) sbias = *(const bf16x4*)(bias + n0 + 4 * tid);
  if (GATED && one_seq && stager)
    sgate = *(const float4*)(epi.gate + (size_t)grow * epi.ld_gate + n0 + 4 * tid);

  const int KT = K / BK;
  gload(0);
  sstore(0);
  if (whole_n && stager) {
    *(float4*)&ebias[4 * tid] =
        float4{(float)sbias[0], (float)sbias[1], (float)sbias[2], (float)sbias[3]};
    if (GATED && one_seq) *(float4*)&egate[4 * tid] = sgate;
  }
  __syncthreads();
  const int fr = lane & 15, fk = (lane >> 4) * 8;
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) gload((kt + 1) * BK);
#pragma unroll
    for (int kk = 0; kk < BK; kk += 32) {
      bf16x8 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *(const bf16x8*)&As[buf][(wm * WM + i * 16 + fr) * LDK + kk + fk];
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *(const bf16x8*)&Bs[buf][(wn * WN + j * 16 + fr) * LDK + kk + fk];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = CT ? __builtin_amdgcn_mfma_f32_16x16x32_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0)
                         : __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < KT) sstore(buf ^ 1);
    __syncthreads();
  }

  if (CT && whole_n) {
    // C^T fragment: lane holds row m = (lane & 15), columns 4*(lane >> 4) + 0..3
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = m0 + wm * WM + i * 16 + fr;
      if (m >= M) continue;
      if constexpr (KIND == EPI_RESID || KIND == EPI_RESID_GATED) {
        // this row's residual values fetched together, then updated
        float4 xl[TN];
#pragma unroll
        for (int j = 0; j < TN; ++j)
          xl[j] = *(const float4*)(epi.x + (size_t)m * epi.ldx + n0 + wn * WN + j * 16 + (lane >> 4) * 4);
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int col = wn * WN + j * 16 + (lane >> 4) * 4;
          const float4 b4 = *(const float4*)&ebias[col];
          float4 g4 = float4{1.f, 1.f, 1.f, 1.f};
          if (GATED) {
            g4 = one_seq ? *(const float4*)&egate[col]
                         : *(const float4*)(epi.gate + (size_t)epi.map.modrow[seq_of_row(epi.map, m)] *
                                                           epi.ld_gate + n0 + col);
          }
          float4 x4 = xl[j];
          x4.x += g4.x * (acc[i][j][0] + b4.x);
          x4.y += g4.y * (acc[i][j][1] + b4.y);
          x4.z += g4.z * (acc[i][j][2] + b4.z);
          x4.w += g4.w * (acc[i][j][3] + b4.w);
          *(float4*)(epi.x + (size_t)m * epi.ldx + n0 + col) = x4;
          if (epi.xb) {
            bf16x4 w{(bf16)x4.x, (bf16)x4.y, (bf16)x4.z, (bf16)x4.w};
            *(bf16x4*)(epi.xb + (size_t)m * epi.ldx + n0 + col) = w;
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int col = wn * WN + j * 16 + (lane >> 4) * 4;
          const float4 b4 = *(const float4*)&ebias[col];
          const float v[4] = {acc[i][j][0] + b4.x, acc[i][j][1] + b4.y, acc[i][j][2] + b4.z,
                              acc[i][j][3] + b4.w};
          epi_store4<EK>(epi, m, n0 + col, v);
        }
      }
    }
  } else if (CT) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = m0 + wm * WM + i * 16 + fr;
      if (m >= M) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int nb = n0 + wn * WN + j * 16 + (lane >> 4) * 4;
        if (vec_ok && nb + 3 < N) {
          const bf16x4 b4 = PART ? bf16x4{} : *(const bf16x4*)(bias + nb);
          const float v[4] = {acc[i][j][0] + (float)b4[0], acc[i][j][1] + (float)b4[1],
                              acc[i][j][2] + (float)b4[2], acc[i][j][3] + (float)b4[3]};
          epi_store4<EK>(epi, m, nb, v);
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (nb + r < N)
              epi_apply<bf16>(epi, EK, m, nb + r, acc[i][j][r] + (PART ? 0.f : (float)bias[nb + r]));
        }
      }
    }
  } else if (KIND == EPI_SPLIT_VT && whole_n && m0 + BM <= M && n0 >= epi.vcol0) {
    // a whole V tile: four consecutive tokens of one V column per store
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + wn * WN + j * 16 + fr;
      const float b = ebias[n - n0];
      bf16* vt = epi.vt + (size_t)(n - epi.vcol0) * epi.ldvt;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int mb = m0 + wm * WM + i * 16 + (lane >> 4) * 4;
        bf16x4 v4;
#pragma unroll
        for (int r = 0; r < 4; ++r) v4[r] = (bf16)(acc[i][j][r] + b);
        *(bf16x4*)(vt + mb) = v4;
      }
    }
  } else if (KIND == EPI_SPLIT_VT && whole_n && m0 + BM <= M && n0 + BN <= epi.vcol0) {
    // a whole q|k tile: no per-element bounds or column-range tests (the
    // query columns scaled exactly as epi_apply scales them)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + wn * WN + j * 16 + fr;
      const float b = ebias[n - n0];
      const float qs = n < epi.qcols ? epi.qscale : 1.f;
      bf16* o = (bf16*)epi.out + n;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int mb = m0 + wm * WM + i * 16 + (lane >> 4) * 4;
#pragma unroll
        for (int r = 0; r < 4; ++r) o[(size_t)(mb + r) * epi.ldo] = (bf16)((acc[i][j][r] + b) * qs);
      }
    }
  } else {
    // C fragment: lane holds column (lane & 15), rows 4*(lane >> 4) + 0..3
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + wn * WN + j * 16 + fr;
      if (n >= N) continue;
      const float b = whole_n ? ebias[n - n0] : (float)bias[n];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int mb = m0 + wm * WM + i * 16 + (lane >> 4) * 4;
        if (KIND == EPI_SPLIT_VT && n >= epi.vcol0 && mb + 3 < M) {
          // four consecutive tokens of one V column: one 8-byte store into V^T
          bf16x4 v4;
#pragma unroll
          for (int r = 0; r < 4; ++r) v4[r] = (bf16)(acc[i][j][r] + b);
          *(bf16x4*)(epi.vt + (size_t)(n - epi.vcol0) * epi.ldvt + mb) = v4;
          continue;
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = mb + r;
          if (m < M) epi_apply<bf16>(epi, KIND, m, n, acc[i][j][r] + b);
        }
      }
    }
  }
}

template <int BM, int BN, int WGM, int KIND>
__global__ __launch_bounds__(256, 1) void gemm_bf16_kernel(
    const bf16* __restrict__ A, int lda, const bf16* __restrict__ W, int ldw,
    const bf16* __restrict__ bias, int M, int N, int K, Epi epi, int tiles_n, int vec_ok) {
  // split-K: workgroup row blockIdx.y takes K columns [y K, (y+1) K) and
  // writes its partial sums to slice y of the fp32 output
  if (KIND == EPI_PARTIAL) {
    A += (size_t)blockIdx.y * K;
    W += (size_t)blockIdx.y * K;
    epi.out = (float*)epi.out + (size_t)blockIdx.y * M * epi.ldo;
  }
  gemm_bf16_body<BM, BN, WGM, KIND>(A, lda, W, ldw, bias, M, N, K, epi, tiles_n, vec_ok,
                                    xcd_remap(blockIdx.x, gridDim.x));
}

// One launch for several GEMMs that share A and the shape: group blockIdx.y
// takes its weight, bias and output pointers from the table.  Each tile is
// computed exactly as by gemm_bf16_kernel.
template <int BM, int BN, int WGM, int KIND>
__global__ __launch_bounds__(256, 1) void gemm_bf16_group_kernel(
    const bf16* __restrict__ A, int lda, PtrGroup g, int ldw, int M, int N, int K, Epi epi,
    int tiles_n, int vec_ok) {
  const int grp = blockIdx.y;
  epi.out = g.out[grp];
  epi.vt = g.vt[grp];
  gemm_bf16_body<BM, BN, WGM, KIND>(A, lda, (const bf16*)g.W[grp], ldw, (const bf16*)g.bias[grp],
                                    M, N, K, epi, tiles_n, vec_ok,
                                    xcd_remap(blockIdx.x, gridDim.x));
}

template <int BM, int BN, int WGM>
static hipError_t gemm_bf16_dispatch(const bf16* A, int lda, const bf16* W, int ldw,
                                     const bf16* bias, int M, int N, int K, int kind,
                                     const Epi& epi, int vec_ok, hipStream_t st, int splits = 1) {
  const int tn = (N + BN - 1) / BN, tm = (M + BM - 1) / BM;
  dim3 grid(tm * tn, splits), block(256);
#define T2I_GEMM_CASE(K_)                                                                       \
  case K_:                                                                                      \
    hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, WGM, K_>), grid, block, 0, st, A, lda, W, ldw, \
                       bias, M, N, K, epi, tn, vec_ok);                                         \
    break;
  switch (kind) {
    T2I_GEMM_CASE(EPI_STORE)
    T2I_GEMM_CASE(EPI_GELU)
    T2I_GEMM_CASE(EPI_SILU)
    T2I_GEMM_CASE(EPI_RESID)
    T2I_GEMM_CASE(EPI_RESID_GATED)
    T2I_GEMM_CASE(EPI_SPLIT_VT)
    T2I_GEMM_CASE(EPI_STORE_F32)
    T2I_GEMM_CASE(EPI_PARTIAL)
    default: return hipErrorInvalidValue;
  }
#undef T2I_GEMM_CASE
  return hipGetLastError();
}

// Split-K reduction: y = bias + sum over slices (fixed order), then the
// epilogue; four consecutive columns per thread.
template <int KIND>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part,
                                                            int splits, const bf16* __restrict__ bias,
                                                            int M, int N, Epi epi, int vec_ok) {
  const int nq = (N + 3) / 4;
  const long total = (long)M * nq;
  const size_t slice = (size_t)M * N;
  for (long i = blockIdx.x * 256L + threadIdx.x; i < total; i += (long)gridDim.x * 256) {
    const int m = (int)(i / nq), nb = (int)(i - (long)m * nq) * 4;
    const float* p = part + (size_t)m * N + nb;
    if (vec_ok && nb + 3 < N && KIND != EPI_SPLIT_VT) {
      const bf16x4 b4 = *(const bf16x4*)(bias + nb);
      float v[4] = {(float)b4[0], (float)b4[1], (float)b4[2], (float)b4[3]};
      for (int z = 0; z < splits; ++z) {
        const float4 q = *(const float4*)(p + z * slice);
        v[0] += q.x;
        v[1] += q.y;
        v[2] += q.z;
        v[3] += q.w;
      }
      epi_store4<KIND>(epi, m, nb, v);
    } else {
      for (int r = 0; r < 4 && nb + r < N; ++r) {
        float v = (float)bias[nb + r];
        for (int z = 0; z < splits; ++z) v += p[z * slice + r];
        epi_apply<bf16>(epi, KIND, m, nb + r, v);
      }
    }
  }
}

// Number of K slices (1 = no split) for a layer whose caller allows
// splitting: narrow outputs (N <= 4096) against K >= 2048, one slice per
// 1024 columns, at most 4.  It depends on the layer's shape only, never on
// M, so a row's result does not depend on how many rows share the launch.
static int splitk_factor(int N, int K) {
  if (N > 4096 || K < 2048) return 1;
  int s = std::min(4, K / 1024);
  while (s > 1 && K % (64 * s) != 0) --s;
  return s;
}

hipError_t launch_gemm_bf16(const bf16* A, int lda, const bf16* W, int ldw, const bf16* bias,
                            int M, int N, int K, int kind, const Epi& epi, float* splitk_ws,
                            size_t splitk_floats, hipStream_t st) {
  if (M <= 0 || N <= 0) return hipSuccess;
  auto al = [](const void* p, int a) { return ((uintptr_t)p % a) == 0; };
  const int vec_ok = (epi.ldo % 4 == 0) && (epi.ldx % 4 == 0) && (epi.ld_gate % 4 == 0) &&
                     al(bias, 8) && al(epi.out, kind == EPI_STORE_F32 ? 16 : 8) &&
                     al(epi.x, 16) && al(epi.xb, 8) && al(epi.gate, 16);
  // Tile choice.  Large M: 256-row tiles fed by direct HBM->LDS loads
  // (gemm_dma.hip).  The DiT widths 1152, 2304, 3456 and 4608 are multiples of
  // 144, so at M = 8192 the layers launch 256 / 512 / 768 / 1024 tiles --
  // whole rounds on 256 CUs at one workgroup each; widths that are multiples
  // of 128 take 192- or 128-wide tiles.  Otherwise 128 x 144 or 128 x 128
  // register-staged tiles (the faster ones at M ~ 1000 measured), with K
  // split over several workgroups when there are too few tiles to fill the
  // chip (e.g. the 512-row text stream against K = 3072 or 12288).
  // (the direct-load kernels address each operand with 32-bit byte offsets)
  const bool dma_fits = (size_t)2 * M * lda < 0x7fffffff && (size_t)2 * N * ldw < 0x7fffffff;
  if (M >= 2048 && (N % 144 == 0 || N % 128 == 0) && kind != EPI_SILU && dma_fits)
    return launch_gemm_dma(A, lda, W, ldw, bias, M, N, K, kind, epi, vec_ok, st);
  const int splits = splitk_ws ? splitk_factor(N, K) : 1;
  if (splits == 1 && N % 144 == 0 && K % 64 == 0 && kind != EPI_SILU && dma_fits && M >= 64)
    return launch_gemm_dma_small(A, lda, W, ldw, bias, M, N, K, kind, epi, vec_ok, st);
  if (splits > 1 && (size_t)splits * M * N <= splitk_floats && kind != EPI_SILU) {
    Epi pe;
    std::memset(&pe, 0, sizeof(pe));
    pe.out = splitk_ws;
    pe.ldo = N;
    const int pvec = N % 4 == 0;
    // 64 x 64 tiles where 128-row tiles would leave most CUs idle (the
    // caption projection of one request: 120 rows); same K order, same sums
    const long t128 = (long)((M + 127) / 128) * ((N + (N % 144 == 0 ? 143 : 127)) /
                                                  (N % 144 == 0 ? 144 : 128));
    hipError_t err =
        t128 * splits < 256
            ? gemm_bf16_dispatch<64, 64, 2>(A, lda, W, ldw, bias, M, N, K / splits, EPI_PARTIAL,
                                            pe, pvec, st, splits)
        : N % 144 == 0
            ? gemm_bf16_dispatch<128, 144, 4>(A, lda, W, ldw, bias, M, N, K / splits, EPI_PARTIAL,
                                              pe, pvec, st, splits)
            : gemm_bf16_dispatch<128, 128, 2>(A, lda, W, ldw, bias, M, N, K / splits, EPI_PARTIAL,
                                              pe, pvec, st, splits);
    if (err != hipSuccess) return err;
    const long work = (long)M * ((N + 3) / 4);
    const int grid = (int)std::min<long>((work + 255) / 256, 4096);
#define T2I_RED_CASE(K_)                                                                   \
  case K_:                                                                                 \
    hipLaunchKernelGGL(splitk_reduce_kernel<K_>, dim3(grid), dim3(256), 0, st, splitk_ws, \
                       splits, bias, M, N, epi, vec_ok && pvec);                           \
    break;
    switch (kind) {
      T2I_RED_CASE(EPI_STORE)
      T2I_RED_CASE(EPI_GELU)
      T2I_RED_CASE(EPI_RESID)
      T2I_RED_CASE(EPI_RESID_GATED)
      T2I_RED_CASE(EPI_SPLIT_VT)
      T2I_RED_CASE(EPI_STORE_F32)
      default: return hipErrorInvalidValue;
    }
#undef T2I_RED_CASE
    return hipGetLastError();
  }
  // 128-row tiles unless they would leave CUs idle (e.g. 1024 rows x 1152
  // columns = 64 tiles); 64 x 64 tiles then (same K order, same results)
  const long tiles128 = (long)((M + 127) / 128) * ((N + (N % 144 == 0 ? 143 : 127)) /
                                                    (N % 144 == 0 ? 144 : 128));
  if (tiles128 < 256)
    return gemm_bf16_dispatch<64, 64, 2>(A, lda, W, ldw, bias, M, N, K, kind, epi, vec_ok, st);
  if (N % 144 == 0)
    return gemm_bf16_dispatch<128, 144, 4>(A, lda, W, ldw, bias, M, N, K, kind, epi, vec_ok, st);
  return gemm_bf16_dispatch<128, 128, 2>(A, lda, W, ldw, bias, M, N, K, kind, epi, vec_ok, st);
}

bool gemm_bf16_groupable(int M, int N, int kind) {
  // the shapes launch_gemm_bf16 runs on register-staged tiles without split-K
  return M > 0 && N > 0 && !(M >= 2048 && (N % 144 == 0 || N % 128 == 0) && kind != EPI_SILU) &&
         (kind == EPI_STORE || kind == EPI_SPLIT_VT);
}

hipError_t launch_gemm_bf16_group(const bf16* A, int lda, const PtrGroup& g, int groups, int ldw,
                                  int M, int N, int K, int kind, const Epi& epi, hipStream_t st) {
  if (groups <= 0) return hipSuccess;
  if (groups > kMaxGroups || !gemm_bf16_groupable(M, N, kind)) return hipErrorInvalidValue;
  auto al = [](const void* p, int a) { return ((uintptr_t)p % a) == 0; };
  int vec_ok = (epi.ldo % 4 == 0) && (epi.ldx % 4 == 0) && (epi.ld_gate % 4 == 0);
  for (int i = 0; i < groups; ++i)
    vec_ok = vec_ok && al(g.bias[i], 8) && al(g.out[i], 8);
  dim3 block(256);
#define T2I_GRP(BM_, BN_, WGM_, K_)                                                          \
  {                                                                                          \
    const int tn = (N + BN_ - 1) / BN_, tm = (M + BM_ - 1) / BM_;                            \
    hipLaunchKernelGGL((gemm_bf16_group_kernel<BM_, BN_, WGM_, K_>), dim3(tm * tn, groups),  \
                       block, 0, st, A, lda, g, ldw, M, N, K, epi, tn, vec_ok);              \
  }
  if (N % 144 == 0) {
    if (kind == EPI_STORE) T2I_GRP(128, 144, 4, EPI_STORE) else T2I_GRP(128, 144, 4, EPI_SPLIT_VT)
  } else {
    if (kind == EPI_STORE) T2I_GRP(128, 128, 2, EPI_STORE) else T2I_GRP(128, 128, 2, EPI_SPLIT_VT)
  }
#undef T2I_GRP
  return hipGetLastError();
}

// ---------------------------------------------------------------------------

template <typename TW, int KIND>
__global__ __launch_bounds__(256) void gemm_f32_kernel(
    const float* __restrict__ A, int lda, const TW* __restrict__ W, int ldw,
    const TW* __restrict__ bias, int M, int N, int K, Epi epi) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ float As[BK][BM + 4];
  __shared__ float Bs[BK][BN + 4];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;

  for (int k0 = 0; k0 < K; k0 += BK) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = tid + 256 * i, r = idx >> 4, kk = idx & 15;
      const int m = m0 + r, n = n0 + r, k = k0 + kk;
      As[kk][r] = (m < M && k < K) ? A[(size_t)m * lda + k] : 0.f;
      Bs[kk][r] = (n < N && k < K) ? to_f32(W[(size_t)n * ldw + k]) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n < N) epi_apply<float>(epi, KIND, m, n, acc[i][j] + to_f32(bias[n]));
    }
  }
}

// ---------------------------------------------------------------------------
// Small-M linear layer (conditioning: timestep MLP and adaLN table, M = number
// of timesteps).  HBM-bound on the weights: each wave owns 4 output columns,
// lanes stream 16-byte chunks of the 4 weight rows once, multiply them with up
// to MT activation rows (fp32, L2-resident), and reduce across the wave.
// Weight reads are contiguous 1 KB per wave instruction.

template <typename TW, int MT, int KIND>
__device__ __forceinline__ void linear_rows_body(const float* __restrict__ A, int lda,
                                                 const TW* __restrict__ W, int ldw,
                                                 const TW* __restrict__ bias, int M, int N, int K,
                                                 const Epi& epi) {
  constexpr int NC = 4;
  const int lane = threadIdx.x & 63;
  const int n0 = (blockIdx.y * 4 + (threadIdx.x >> 6)) * NC;
  const int m0 = blockIdx.x * MT;
  if (n0 >= N) return;
  const int mt = min(MT, M - m0);
  float acc[MT][NC];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int j = 0; j < NC; ++j) acc[m][j] = 0.f;
  for (int k = lane * 8; k < K; k += 64 * 8) {
    float wv[NC][8];
#pragma unroll
    for (int j = 0; j < NC; ++j) {
      const int n = min(n0 + j, N - 1);
      const TW* wp = W + (size_t)n * ldw + k;
      if constexpr (sizeof(TW) == 2) {
        const bf16x8 v = *(const bf16x8*)wp;
#pragma unroll
        for (int e = 0; e < 8; ++e) wv[j][e] = (float)v[e];
      } else {
        const float4 a = *(const float4*)wp, b = *(const float4*)(wp + 4);
        wv[j][0] = a.x; wv[j][1] = a.y; wv[j][2] = a.z; wv[j][3] = a.w;
        wv[j][4] = b.x; wv[j][5] = b.y; wv[j][6] = b.z; wv[j][7] = b.w;
      }
    }
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      if (m < mt) {
        const float* ap = A + (size_t)(m0 + m) * lda + k;
        const float4 a = *(const float4*)ap, b = *(const float4*)(ap + 4);
        const float av[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
        for (int j = 0; j < NC; ++j)
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[m][j] = fmaf(av[e], wv[j][e], acc[m][j]);
      }
    }
  }
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    if (m >= mt) break;
#pragma unroll
    for (int j = 0; j < NC; ++j) {
      const float v = wave_sum(acc[m][j]);
      if (lane == 0 && n0 + j < N) epi_apply<float>(epi, KIND, m0 + m, n0 + j, v + to_f32(bias[n0 + j]));
    }
  }
}

template <typename TW, int MT, int KIND>
__global__ __launch_bounds__(256) void linear_rows_kernel(const float* __restrict__ A, int lda,
                                                          const TW* __restrict__ W, int ldw,
                                                          const TW* __restrict__ bias, int M,
                                                          int N, int K, Epi epi) {
  linear_rows_body<TW, MT, KIND>(A, lda, W, ldw, bias, M, N, K, epi);
}

// Several weight matrices against the same rows in one launch: group
// blockIdx.z takes its weight, bias and output from the table.
template <typename TW, int MT, int KIND>
__global__ __launch_bounds__(256) void linear_rows_group_kernel(const float* __restrict__ A,
                                                                int lda, PtrGroup g, int ldw,
                                                                int M, int N, int K, Epi epi) {
  const int grp = blockIdx.z;
  epi.out = g.out[grp];
  linear_rows_body<TW, MT, KIND>(A, lda, (const TW*)g.W[grp], ldw, (const TW*)g.bias[grp], M, N,
                                 K, epi);
}

template <typename TW, int MT>
static hipError_t linear_rows_dispatch(const float* A, int lda, const TW* W, int ldw,
                                       const TW* bias, int M, int N, int K, int kind,
                                       const Epi& epi, hipStream_t st) {
  // consecutive workgroups share weight rows (row passes vary fastest)
  dim3 grid((M + MT - 1) / MT, (N + 15) / 16), block(256);
  switch (kind) {
    case EPI_STORE:
      hipLaunchKernelGGL((linear_rows_kernel<TW, MT, EPI_STORE>), grid, block, 0, st, A, lda, W, ldw, bias, M, N, K, epi);
      break;
    case EPI_SILU:
      hipLaunchKernelGGL((linear_rows_kernel<TW, MT, EPI_SILU>), grid, block, 0, st, A, lda, W, ldw, bias, M, N, K, epi);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_linear_rows_group(const float* A, int lda, const PtrGroup& g, int groups,
                                    int ldw, bool w_bf16, int M, int N, int K, const Epi& epi,
                                    hipStream_t st) {
  if (groups <= 0 || M <= 0 || N <= 0) return hipSuccess;
  if (groups > kMaxGroups || K % 8 || lda % 4 || ldw % 8 || ((uintptr_t)A & 15))
    return hipErrorInvalidValue;
  for (int i = 0; i < groups; ++i)
    if ((uintptr_t)g.W[i] & 15) return hipErrorInvalidValue;
  dim3 grid((M + 7) / 8, (N + 15) / 16, groups), block(256);
  if (w_bf16 && M <= 2) {
    // one step's conditioning rows: a 2-row instance needs fewer registers,
    // so more waves stream weights at once (each row's sums are those of the
    // 8-row instance)
    grid.x = 1;
    hipLaunchKernelGGL((linear_rows_group_kernel<bf16, 2, EPI_STORE>), grid, block, 0, st, A, lda,
                       g, ldw, M, N, K, epi);
  } else if (w_bf16)
    hipLaunchKernelGGL((linear_rows_group_kernel<bf16, 8, EPI_STORE>), grid, block, 0, st, A, lda,
                       g, ldw, M, N, K, epi);
  else
    hipLaunchKernelGGL((linear_rows_group_kernel<float, 8, EPI_STORE>), grid, block, 0, st, A, lda,
                       g, ldw, M, N, K, epi);
  return hipGetLastError();
}

hipError_t launch_linear_rows(const float* A, int lda, const void* W, int ldw, bool w_bf16,
                              const void* bias, int M, int N, int K, int kind, const Epi& epi,
                              hipStream_t st) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if ((kind != EPI_STORE && kind != EPI_SILU) || K % 8 || lda % 4 || ldw % 8 ||
      ((uintptr_t)A & 15) || ((uintptr_t)W & 15))
    return hipErrorInvalidValue;
  if (w_bf16)
    return linear_rows_dispatch<bf16, 8>(A, lda, (const bf16*)W, ldw, (const bf16*)bias, M, N, K, kind, epi, st);
  return linear_rows_dispatch<float, 8>(A, lda, (const float*)W, ldw, (const float*)bias, M, N, K, kind, epi, st);
}

template <typename TW>
static hipError_t gemm_f32_dispatch(const float* A, int lda, const TW* W, int ldw, const TW* bias,
                                    int M, int N, int K, int kind, const Epi& epi, hipStream_t st) {
  dim3 grid((N + 63) / 64, (M + 63) / 64), block(256);
  switch (kind) {
    case EPI_STORE:
      hipLaunchKernelGGL((gemm_f32_kernel<TW, EPI_STORE>), grid, block, 0, st, A, lda, W, ldw, bias, M, N, K, epi);
      break;
    case EPI_GELU:
      hipLaunchKernelGGL((gemm_f32_kernel<TW, EPI_GELU>), grid, block, 0, st, A, lda, W, ldw, bias, M, N, K, epi);
      break;
    case EPI_SILU:
      hipLaunchKernelGGL((gemm_f32_kernel<TW, EPI_SILU>), grid, block, 0, st, A, lda, W, ldw, bias, M, N, K, epi);
      break;
    case EPI_RESID:
      hipLaunchKernelGGL((gemm_f32_kernel<TW, EPI_RESID>), grid, block, 0, st, A, lda, W, ldw, bias, M, N, K, epi);
      break;
    default:
      hipLaunchKernelGGL((gemm_f32_kernel<TW, EPI_RESID_GATED>), grid, block, 0, st, A, lda, W, ldw, bias, M, N, K, epi);
      break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm_f32(const float* A, int lda, const void* W, int ldw, bool w_bf16,
                           const void* bias, int M, int N, int K, int kind, const Epi& epi,
                           hipStream_t st) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (w_bf16)
    return gemm_f32_dispatch<bf16>(A, lda, (const bf16*)W, ldw, (const bf16*)bias, M, N, K, kind, epi, st);
  return gemm_f32_dispatch<float>(A, lda, (const float*)W, ldw, (const float*)bias, M, N, K, kind, epi, st);
}

}  // namespace t2i
