// bf16 MFMA GEMM fed by direct HBM->LDS loads (gfx950 buffer_load_dwordx4 ... lds).
//
// y = A W^T + b for the DiT's projections at large M.  A workgroup owns a
// BM x BN output tile; its waves (WGM x WGN) each own a (BM/WGM) x (BN/WGN)
// quadrant of 16x16 MFMA tiles (v_mfma_f32_16x16x32_bf16, fp32 accumulation).
// K advances 64 at a time through a ring of ST LDS stages (see launch_gemm_dma
// for the tile shapes in use):
//
//   * each stage holds the A rows (BM x 128 B) then the W rows (BN x 128 B);
//     every 1 KB of a stage (8 rows) is filled by ONE wave instruction that
//     moves 16 bytes per lane straight from global memory into LDS -- no
//     registers, no ds_write;
//   * rows are not padded: the 16-byte chunk c of row r sits in slot
//     c ^ ((r >> 1) & 7), so the 16 rows one fragment load touches spread over
//     all 64 banks (rows alternate bank halves; the swizzle separates the 8
//     rows of each half);
//   * ST-1 tiles are in flight while one is consumed: per K step a wave waits
//     until only its loads of the younger tiles are outstanding (vmcnt),
//     meets the other waves at one barrier, issues the loads of tile t+ST-1
//     into the stage everybody finished with, and runs its MFMAs;
//   * every wave issues the same number of load instructions per tile
//     (waves with fewer blocks repeat their last one, which rewrites identical
//     bytes), so the vmcnt thresholds are compile-time constants;
//   * loads address A and W through buffer resources (per-lane 32-bit byte
//     offsets, the K position as scalar offset; the caller keeps both
//     operands below 2^31 bytes).  The buffer form rather than the global
//     one because the compiler tracks it by vmcnt alone: an outstanding
//     global-form LDS load counts as an out-of-order LDS event, after which
//     every fragment read is drained with lgkmcnt(0) instead of counted.
//
// The epilogue is the one of gemm.hip: C^T fragments (operands swapped) give a
// lane four consecutive output columns of one row, stored with one 8-byte
// (bf16) or 16-byte (fp32 residual) access; the split q|k|v store keeps the C
// layout and writes V^T four tokens at a time.
#include <algorithm>

#include "t2i_internal.h"
#include "xattn_tile.h"

namespace t2i {

__device__ __forceinline__ int xcd_remap_dma(int b, int nb) {
  const int q = nb >> 3, r = nb & 7;
  const int x = b & 7, j = b >> 3;
  return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + j;
}

// s_waitcnt with only vmcnt constrained (gfx9 encoding: vmcnt low bits [3:0],
// high bits [15:14]; expcnt [6:4] and lgkmcnt [11:8] left at their maximum).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// one 16-byte-per-lane buffer load into LDS at the wave-uniform address lds
template <int AUX>
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, char* lds, uint32_t voff, int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16,
                                           voff, soff, 0, AUX);
}

// wait until at most `younger` load rounds of BPW instructions each are
// outstanding (younger <= 5; compile-time counts)
template <int BPW>
__device__ __forceinline__ void wait_rounds(int younger) {
  switch (younger) {
    case 0: wait_vmcnt<0>(); break;
    case 1: wait_vmcnt<BPW>(); break;
    case 2: wait_vmcnt<(2 * BPW < 64 ? 2 * BPW : 0)>(); break;
    case 3: wait_vmcnt<(3 * BPW < 64 ? 3 * BPW : 0)>(); break;
    case 4: wait_vmcnt<(4 * BPW < 64 ? 4 * BPW : 0)>(); break;
    default: wait_vmcnt<(5 * BPW < 64 ? 5 * BPW : 0)>(); break;
  }
}

__device__ __forceinline__ void block_barrier() {
  // this wave's LDS reads are complete (a stage may be refilled right after
  // the barrier), then a plain s_barrier: no release fence, which would wait
  // for every outstanding global load, and a compiler barrier for memory ops.
  // The wait is the builtin, so that the compiler's wait-count tracking knows
  // nothing is pending after it.
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0), vmcnt / expcnt untouched
  asm volatile("s_barrier" ::: "memory");
}

// xpre: this fragment's residual values when already fetched; gated updates
// take the gate values g4 when have_g, else read them here
template <int KIND>
__device__ __forceinline__ void dma_epi4(const Epi& e, int m, int nb, const float v[4],
                                         const float4* xpre = nullptr, bool have_g = false,
                                         float4 g4 = float4{1.f, 1.f, 1.f, 1.f}) {
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
    if (KIND == EPI_RESID_GATED && !have_g)
      g4 = *(const float4*)(e.gate + (size_t)e.map.modrow[seq_of_row(e.map, m)] * e.ld_gate + nb);
    float4* xp = (float4*)(e.x + (size_t)m * e.ldx + nb);
    float4 x4 = xpre ? *xpre : *xp;
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

// No cross-attention after the projection.
struct XNone {
  static constexpr bool on = false;
};

// XT: XNone, or XAttnArgs for the cross-attention query projection with the
// cross-attention fused in (256 x 144 tiles, EPI_STORE; launch_gemm_xattn)
template <int BM, int BN, int WGM, int WGN, int ST, int KIND, int AUX, class XT>
__global__ __launch_bounds__(64 * WGM * WGN, 1) void gemm_dma_kernel(
    const bf16* __restrict__ A, int lda, const bf16* __restrict__ W, int ldw,
    const bf16* __restrict__ bias, int M, int N, int K, Epi epi, int tiles_n, int group_m,
    int vec_ok, XT xa) {
  constexpr int NW = WGM * WGN;
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int ABLK = BM / 8, BBLK = BN / 8, TBLK = ABLK + BBLK;   // 1-KB blocks per stage
  constexpr int BPW = (TBLK + NW - 1) / NW;                       // load instructions per wave
  constexpr int STAGE = (BM + BN) * 64;                            // bf16 elements per stage
  constexpr bool CT = KIND != EPI_SPLIT_VT;
  static_assert(BM % 8 == 0 && BN % 8 == 0 && WM % 16 == 0 && WN % 16 == 0, "tile shape");
  static_assert(ST >= 2 && ST <= 7 && (ST - 2) * BPW < 64, "stages");
  static_assert(ABLK % NW == 0, "A / W blocks split evenly over the load rounds");
  // the stage ring, then the epilogue's fp32 bias and gate rows (one LDS
  // object: with several, the compiler makes every fragment read wait for
  // all outstanding tile loads)
  constexpr bool GATED = KIND == EPI_RESID_GATED;
  __shared__ __attribute__((aligned(1024))) bf16 smem[ST * STAGE + (GATED ? 4 : 2) * BN];
  float* const ebias = (float*)(smem + ST * STAGE);
  float* const egate = ebias + BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  // tile order: the tiles of one XCD are consecutive; within that range they
  // walk group_m row blocks down before moving one column block right, so the
  // workgroups resident on an XCD share both A rows and W rows in its L2
  const int tile = xcd_remap_dma(blockIdx.x, gridDim.x);
  const int tiles_m = (M + BM - 1) / BM;
  const int per_group = group_m * tiles_n, grp = tile / per_group;
  const int first = grp * group_m, rows_in = min(tiles_m - first, group_m);
  const int in_grp = tile - grp * per_group;
  const int m0 = (first + in_grp % rows_in) * BM, n0 = (in_grp / rows_in) * BN;

  // this lane's byte offset of every block it loads, from A or W (the k
  // position is added per tile as the scalar offset); load round i reads A
  // while i < ABLK / NW
  uint32_t src[BPW];
  int dst[BPW];   // byte offset of the block inside a stage (wave-uniform)
#pragma unroll
  for (int i = 0; i < BPW; ++i) {
    int b = wave + i * NW;
    if (b >= TBLK) b -= NW;               // repeat this wave's previous block
    const int lr = (b < ABLK ? b : b - ABLK) * 8 + (lane >> 3);   // row within A or W tile
    const int c = (lane & 7) ^ ((lr >> 1) & 7);                   // logical chunk of this slot
    src[i] = 2u * (uint32_t)(i < ABLK / NW ? min(m0 + lr, M - 1) * lda + c * 8
                                           : min(n0 + lr, N - 1) * ldw + c * 8);
    dst[i] = b * 1024;
  }
  const __amdgpu_buffer_rsrc_t ra =
      __builtin_amdgcn_make_buffer_rsrc((void*)A, 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rw =
      __builtin_amdgcn_make_buffer_rsrc((void*)W, 0, 0x7fffffff, 0x00020000);
  auto issue = [&](int t, int stage) {
    const int kb = t * 128;   // byte offset of the tile's 64 k values
#pragma unroll
    for (int i = 0; i < BPW; ++i)
      dma16<AUX>(i < ABLK / NW ? ra : rw, (char*)smem + stage * STAGE * 2 + dst[i], src[i], kb);
  };

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int fr = lane & 15, g = lane >> 4;
  // byte offset of a fragment row's 16-byte chunk c in the swizzled layout
  auto frag = [&](const bf16* base, int row, int c) {
    return *(const bf16x8*)((const char*)base + row * 128 + ((c ^ ((row >> 1) & 7)) << 4));
  };
  auto compute = [&](int stage) {
    const bf16* sA = smem + stage * STAGE;
    const bf16* sB = sA + BM * 64;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      bf16x8 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) af[i] = frag(sA, wm * WM + i * 16 + fr, kk * 4 + g);
#pragma unroll
      for (int j = 0; j < TN; ++j) bfr[j] = frag(sB, wn * WN + j * 16 + fr, kk * 4 + g);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = CT ? __builtin_amdgcn_mfma_f32_16x16x32_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0)
                         : __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
  };

  // Epilogue operands of a tile that is whole in N: its BN bias values and,
  // for a gated update whose rows all belong to one sequence, its BN gate
  // values.  The first BN / 4 threads fetch them now, ahead of every tile
  // load (so the vmcnt thresholds below, which count younger loads, stay
  // exact), and put them in LDS after the main loop; the epilogue then reads
  // LDS only and its stores never wait behind a global load.
  const bool whole_n = vec_ok && n0 + BN <= N;
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

  // Residual updates with small per-wave tiles read this lane's fp32
  // residual values before the main loop: all workgroups of such a launch
  // reach the epilogue together, and its HBM reads would otherwise come after
  // the loop instead of under it.  Issued before the first tile loads, so the
  // vmcnt thresholds below (which count younger loads) stay exact.  (Measured
  // faster for the gated updates -- out-projection 45.5 -> 40.2 us, fc2 --
  // and, once the epilogue read its bias from LDS, for the plain one after
  // cross-attention too: 37.8 -> 35.5 us.)
  constexpr bool PREX = CT && (KIND == EPI_RESID_GATED || KIND == EPI_RESID) && TM * TN <= 18;
  float4 xpre[PREX ? TM : 1][PREX ? TN : 1];
  if constexpr (PREX) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int m = m0 + wm * WM + i * 16 + fr, nb = n0 + wn * WN + j * 16 + g * 4;
        xpre[i][j] = float4{0.f, 0.f, 0.f, 0.f};
        if (m < M && vec_ok && nb + 3 < N)
          xpre[i][j] = *(const float4*)(epi.x + (size_t)m * epi.ldx + nb);
      }
  }

  // Cross-attention after the projection (XT = XAttnArgs): this tile's two
  // heads (72 columns each) attend to the text of the sequence its rows
  // belong to.  The text's K / V^T tiles go into the first XKV bytes of the
  // ring once the last K step's barrier has passed (that step reads the last
  // stage, the host makes K / 64 a multiple of ST), so they load under that
  // step's MFMAs; the queries are staged at XQ_OFF after the loop.
  constexpr int XHD = 72;
  using XX = XTile<XHD>;
  constexpr int XKV = 4 * (XX::KSTAGE + XX::VSTAGE);
  constexpr int XQ_OFF = ((XKV + (XX::HDO - XX::VROWS) * 128) + 1023) / 1024 * 1024;
  auto xk = [&](int hd, int t) { return (char*)smem + (2 * hd + t) * (XX::KSTAGE + XX::VSTAGE); };
  auto xv = [&](int hd, int t) { return xk(hd, t) + XX::KSTAGE; };
  int xs = 0;
  if constexpr (XT::on) {
    static_assert(BM == 256 && BN == 2 * XHD && WGN == 1 && (ST - 1) * STAGE * 2 >= XKV &&
                      XQ_OFF + NW * 32 * BN * 2 <= ST * STAGE * 2,
                  "fused cross-attention tile");
#pragma unroll 1
    for (int i = 1; i < xa.n; ++i) xs += (m0 >= xa.q_start[i]) ? 1 : 0;
  }
  auto xattn_prefetch = [&]() {
    if constexpr (XT::on) {
      const int nkeys = xa.k_len[xs], k0 = xa.k_start[xs];
      const int nt = (nkeys + XX::BKV - 1) / XX::BKV;
      const __amdgpu_buffer_rsrc_t rk =
          __builtin_amdgcn_make_buffer_rsrc((void*)xa.K, 0, 0x7fffffff, 0x00020000);
      const __amdgpu_buffer_rsrc_t rv =
          __builtin_amdgcn_make_buffer_rsrc((void*)xa.Vt, 0, 0x7fffffff, 0x00020000);
      // (head, tile, instruction) triples spread over the waves
#pragma unroll 1
      for (int idx = __builtin_amdgcn_readfirstlane(wave); idx < 4 * XX::NI; idx += NW) {
        const int hd = idx / (2 * XX::NI), t = (idx / XX::NI) % 2, i = idx % XX::NI;
        if (t < nt)
          xattn_dma<XHD>(rk, rv, i, k0 + t * XX::BKV, k0 + nkeys, n0 / XHD + hd, xa.ldk, xa.ldvt,
                         xk(hd, t), xv(hd, t));
      }
#pragma unroll
      for (int f = 0; f < 4; ++f) xattn_ones<XHD>(xv(f >> 1, f & 1), tid, NW * 64);
    }
  };

  const int KT = K / 64;
  // The small-M tiles (fewer rows per wave, spare registers) meet at the
  // barrier for stage t + 1 halfway through stage t: the fragment reads of a
  // half-step are then issued one half-step ahead and their LDS latency hides
  // under the MFMAs instead of opening each K step (same MFMAs in the same
  // order).  The stage of step t is refilled at that barrier (every wave has
  // its fragments in registers by then).  Measured at 1024 rows: out-
  // projection 20.1 -> 18.6 us, fc2 45.9 -> 42.2, 194 -> 202 steps/s; slower
  // for the 256-row tiles (cross query 26.7 -> 28.2 us), which keep the plain
  // loop.
  constexpr int REGS = TM * TN * 4 + 2 * (TM + TN) * 4 + (PREX ? TM * TN * 4 : 0);
  constexpr bool HALF_STEP = ST >= 3 && BM < 256 && REGS <= 176;
  if constexpr (HALF_STEP) {
    auto read_frags = [&](int slot, int kk, bf16x8 (&af)[TM], bf16x8 (&bfr)[TN]) {
      const bf16* sA = smem + slot * STAGE;
      const bf16* sB = sA + BM * 64;
#pragma unroll
      for (int i = 0; i < TM; ++i) af[i] = frag(sA, wm * WM + i * 16 + fr, kk * 4 + g);
#pragma unroll
      for (int j = 0; j < TN; ++j) bfr[j] = frag(sB, wn * WN + j * 16 + fr, kk * 4 + g);
    };
    auto mma = [&](const bf16x8 (&af)[TM], const bf16x8 (&bfr)[TN]) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = CT ? __builtin_amdgcn_mfma_f32_16x16x32_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0)
                         : __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    };
#pragma unroll
    for (int s = 0; s < ST - 1; ++s)
      if (s < KT) issue(s, s);
    wait_rounds<BPW>(min(ST - 2, KT - 1));   // stage 0 (stages 1 .. ST-2 may fly)
    block_barrier();
    if (ST - 1 < KT) issue(ST - 1, ST - 1);
    bf16x8 a0[TM], b0[TN], a1[TM], b1[TN];
    read_frags(0, 0, a0, b0);
    for (int t0 = 0; t0 < KT; t0 += ST) {
#pragma unroll
      for (int i = 0; i < ST; ++i) {
        const int t = t0 + i;
        if (t >= KT) break;
        read_frags(i, 1, a1, b1);
        mma(a0, b0);
        if (t + 1 < KT) {
          // stage t + 1 landed (stages t + 2 .. t + ST - 1 may fly)
          wait_rounds<BPW>(min(ST - 2, KT - 2 - t));
          block_barrier();
          if (t + ST < KT) issue(t + ST, i);
          read_frags((i + 1) % ST, 0, a0, b0);
        }
        mma(a1, b1);
      }
    }
  } else {
#pragma unroll
    for (int s = 0; s < ST - 1; ++s)
      if (s < KT) issue(s, s);
    for (int t0 = 0; t0 < KT; t0 += ST) {
#pragma unroll
      for (int i = 0; i < ST; ++i) {
        const int t = t0 + i;
        if (t >= KT) break;
        // loads younger than tile t that may stay in flight
        wait_rounds<BPW>(min(ST - 2, KT - 1 - t));
        block_barrier();
        if (t + ST - 1 < KT) issue(t + ST - 1, (i + ST - 1) % ST);
        if (XT::on && t == KT - 1) xattn_prefetch();
        compute(i);
      }
    }
  }

  if (whole_n) {
    if (stager) {
      *(float4*)&ebias[4 * tid] =
          float4{(float)sbias[0], (float)sbias[1], (float)sbias[2], (float)sbias[3]};
      if (GATED && one_seq) *(float4*)&egate[4 * tid] = sgate;
    }
    block_barrier();
  }

  if constexpr (XT::on) {
    // Fused cross-attention (whole tile, whole_n: the host checks).  Each
    // wave rounds its 32 rows of queries exactly as the plain projection
    // stores them (bias, softmax scale, one rounding to bf16) into its part
    // of the ring, then attends with them, head by head, to the text tiles.
    constexpr int QROW = BN * 2;   // staged query row (bytes)
    char* const qst = (char*)smem + XQ_OFF + wave * 32 * QROW;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int col = j * 16 + g * 4;
        const float4 b4 = *(const float4*)&ebias[col];
        const float v[4] = {acc[i][j][0] + b4.x, acc[i][j][1] + b4.y, acc[i][j][2] + b4.z,
                            acc[i][j][3] + b4.w};
        const float qs = n0 + col < epi.qcols ? epi.qscale : 1.f;
        bf16x4 w;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float y = v[r];
          y *= qs;
          w[r] = (bf16)y;
        }
        *(bf16x4*)(qst + (i * 16 + fr) * QROW + col * 2) = w;
      }
    wait_vmcnt<0>();   // this wave's text tile loads
    block_barrier();
    const int nkeys = xa.k_len[xs];
    bool ragged = false;
#pragma unroll
    for (int hd = 0; hd < 2; ++hd)
      ragged = xattn_fix_ragged<XHD>(xv(hd, (nkeys - 1) / XX::BKV), nkeys, tid, NW * 64);
    if (ragged) block_barrier();
    const int ql = lane & 31, hl = lane >> 5;
#pragma unroll 1
    for (int hd = 0; hd < 2; ++hd) {
      bf16x8 qf[XX::DC];
#pragma unroll
      for (int c = 0; c < XX::DC; ++c) {
        const int d = c * 16 + hl * 8;
        qf[c] = d < XHD ? *(const bf16x8*)(qst + ql * QROW + (hd * XHD + d) * 2) : bf16x8{};
      }
      // the head's outputs replace its queries in the wave's rows, then go
      // out along the rows, 16 bytes per lane (faster than the lanes' own
      // 8-byte pieces of 32 rows); the wave's LDS accesses execute in order
      xattn_wave<XHD, true>(xk(hd, 0), xk(hd, 1), xv(hd, 0), xv(hd, 1), nkeys, qf, 1.f, true,
                            [&](int d, bf16x4 w) {
                              *(bf16x4*)(qst + ql * QROW + (hd * XHD + d) * 2) = w;
                            });
      constexpr int CPH = XHD * 2 / 16, NCH = 32 * CPH;   // 16-byte chunks per head row, per wave
#pragma unroll
      for (int c0 = 0; c0 < NCH; c0 += 64) {
        const int c = c0 + lane, row = c / CPH, ch = c - row * CPH;
        if (NCH % 64 == 0 || c < NCH)
          *(uint4*)(xa.O + (size_t)(m0 + wave * 32 + row) * xa.ldo + n0 + hd * XHD + ch * 8) =
              *(const uint4*)(qst + row * QROW + hd * XHD * 2 + ch * 16);
      }
    }
    return;
  }

  if (CT) {
    // Staged stores.  A C^T fragment gives a lane four columns of one row, so
    // direct stores write 16 rows x 32 bytes (bf16) per instruction; the same
    // bytes written as 16-byte chunks along the rows take ~30 % less time (a
    // probe writing a 8192 x 3456 bf16 matrix in 256 x 144 tiles: 17.4 us
    // against 10.7).  So each wave puts its rows, 16 at a time, into its own
    // part of the stage ring (free after the barrier above; one wave's LDS
    // accesses execute in order) and writes them back along the rows.  Every
    // element is computed and rounded as before.  Used for the 256-row tiles
    // (out-projection 41.0 -> 39.6 us at 8192 rows, 73.5 -> 62.0 at 12 032)
    // except 256 x 256 (the joint-attention model's fc1 measured 2.8 %
    // slower), not for the small-M tiles (no gain at 1024 rows).
    constexpr bool STAGED = BM == 256 && BN != 256 && KIND != EPI_STORE_F32 && KIND != EPI_SILU;
    // (16-byte row chunks: row strides and bases must keep them aligned)
    constexpr bool F32O = KIND == EPI_RESID || KIND == EPI_RESID_GATED;
    const bool aligned16 =
        F32O ? ((uintptr_t)epi.x % 16 == 0 && epi.ldx % 4 == 0 &&
                (!epi.xb || ((uintptr_t)epi.xb % 16 == 0 && epi.ldx % 8 == 0)))
             : ((uintptr_t)epi.out % 16 == 0 && epi.ldo % 8 == 0);
    if (STAGED && whole_n && aligned16) {
      constexpr bool F32OUT = KIND == EPI_RESID || KIND == EPI_RESID_GATED;
      constexpr int SROW = WN * (F32OUT ? 4 : 2);   // bytes per staged row
      static_assert(NW * 16 * WN * 4 <= ST * STAGE * 2, "staging fits the ring");
      char* const stg = (char*)smem + wave * 16 * SROW;
      const bool xbw = F32OUT && epi.xb != nullptr;
      // residual values not prefetched: a row's values fetched together
      constexpr bool XL = F32OUT && !PREX;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int mrow0 = m0 + wm * WM + i * 16, m = mrow0 + fr;
        float4 xl[XL ? TN : 1];
        if constexpr (XL) {
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            xl[j] = float4{0.f, 0.f, 0.f, 0.f};
            if (m < M)
              xl[j] = *(const float4*)(epi.x + (size_t)m * epi.ldx + n0 + wn * WN + j * 16 + g * 4);
          }
        }
        bf16x4 xbv[F32OUT ? TN : 1];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int col = wn * WN + j * 16 + g * 4;
          const float4 b4 = *(const float4*)&ebias[col];
          const float v[4] = {acc[i][j][0] + b4.x, acc[i][j][1] + b4.y, acc[i][j][2] + b4.z,
                              acc[i][j][3] + b4.w};
          if constexpr (F32OUT) {
            float4 g4 = float4{1.f, 1.f, 1.f, 1.f};
            if constexpr (GATED) {
              if (one_seq)
                g4 = *(const float4*)&egate[col];
              else if (m < M)
                g4 = *(const float4*)(epi.gate +
                                      (size_t)epi.map.modrow[seq_of_row(epi.map, m)] * epi.ld_gate +
                                      n0 + col);
            }
            float4 x4;
            if constexpr (PREX) x4 = xpre[i][j];
            else x4 = xl[j];
            x4.x += g4.x * v[0];
            x4.y += g4.y * v[1];
            x4.z += g4.z * v[2];
            x4.w += g4.w * v[3];
            *(float4*)(stg + fr * SROW + (j * 16 + g * 4) * 4) = x4;
            xbv[j] = bf16x4{(bf16)x4.x, (bf16)x4.y, (bf16)x4.z, (bf16)x4.w};
          } else {
            bf16x4 w;
            const float qs = KIND == EPI_STORE && n0 + col < epi.qcols ? epi.qscale : 1.f;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              float y = v[r];
              if (KIND == EPI_GELU) y = gelu_tanh(y);
              if (KIND == EPI_STORE) y *= qs;
              w[r] = (bf16)y;
            }
            *(bf16x4*)(stg + fr * SROW + (j * 16 + g * 4) * 2) = w;
          }
        }
        // the 16 rows back along the rows, 16 bytes per lane
        {
          constexpr int CPRW = SROW / 16, NCH = 16 * CPRW;
#pragma unroll
          for (int c0 = 0; c0 < NCH; c0 += 64) {
            const int c = c0 + lane, row = c / CPRW, ch = c - row * CPRW;
            if ((NCH % 64 == 0 || c < NCH) && mrow0 + row < M) {
              const uint4 d = *(const uint4*)(stg + row * SROW + ch * 16);
              if constexpr (F32OUT)
                *(uint4*)(epi.x + (size_t)(mrow0 + row) * epi.ldx + n0 + wn * WN + ch * 4) = d;
              else
                *(uint4*)((bf16*)epi.out + (size_t)(mrow0 + row) * epi.ldo + n0 + wn * WN + ch * 8) = d;
            }
          }
        }
        if (F32OUT && xbw) {
          // the bf16 copy of the residual through the same rows
          constexpr int SROWB = WN * 2, CPRB = SROWB / 16, NCHB = 16 * CPRB;
#pragma unroll
          for (int j = 0; j < TN; ++j)
            *(bf16x4*)(stg + fr * SROWB + (j * 16 + g * 4) * 2) = xbv[j];
#pragma unroll
          for (int c0 = 0; c0 < NCHB; c0 += 64) {
            const int c = c0 + lane, row = c / CPRB, ch = c - row * CPRB;
            if ((NCHB % 64 == 0 || c < NCHB) && mrow0 + row < M) {
              const uint4 d = *(const uint4*)(stg + row * SROWB + ch * 16);
              *(uint4*)(epi.xb + (size_t)(mrow0 + row) * epi.ldx + n0 + wn * WN + ch * 8) = d;
            }
          }
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int m = m0 + wm * WM + i * 16 + fr;
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int nb = n0 + wn * WN + j * 16 + g * 4;
          if (vec_ok && nb + 3 < N) {
            const bf16x4 b4 = *(const bf16x4*)(bias + nb);
            const float v[4] = {acc[i][j][0] + (float)b4[0], acc[i][j][1] + (float)b4[1],
                                acc[i][j][2] + (float)b4[2], acc[i][j][3] + (float)b4[3]};
            if constexpr (PREX) dma_epi4<KIND>(epi, m, nb, v, &xpre[i][j]);
            else dma_epi4<KIND>(epi, m, nb, v);
          } else {
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (nb + r < N) epi_apply<bf16>(epi, KIND, m, nb + r, acc[i][j][r] + (float)bias[nb + r]);
          }
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
        const int mb = m0 + wm * WM + i * 16 + g * 4;
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
        const int mb = m0 + wm * WM + i * 16 + g * 4;
#pragma unroll
        for (int r = 0; r < 4; ++r) o[(size_t)(mb + r) * epi.ldo] = (bf16)((acc[i][j][r] + b) * qs);
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + wn * WN + j * 16 + fr;
      if (n >= N) continue;
      const float b = whole_n ? ebias[n - n0] : (float)bias[n];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int mb = m0 + wm * WM + i * 16 + g * 4;
        if (KIND == EPI_SPLIT_VT && n >= epi.vcol0 && mb + 3 < M) {
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

// s_waitcnt vmcnt(n) for a wave-uniform n known only at run time; n > 15
// waits for vmcnt(15), which is stricter
__device__ __forceinline__ void wait_vmcnt_dyn15(int n) {
  switch (n) {
#define T2I_W(N_) case N_: wait_vmcnt<N_>(); break;
    T2I_W(0) T2I_W(1) T2I_W(2) T2I_W(3) T2I_W(4) T2I_W(5) T2I_W(6) T2I_W(7)
    T2I_W(8) T2I_W(9) T2I_W(10) T2I_W(11) T2I_W(12) T2I_W(13) T2I_W(14)
#undef T2I_W
    default: wait_vmcnt<15>(); break;
  }
}

// The split q|k|v projection when it takes several rounds of 256 x 144 tiles
// (the 1024-px guided step: 768 tiles, three per CU).  In gemm_dma_kernel
// every workgroup of a round reaches its epilogue at the same time and the
// MFMA pipes idle through it (~6 us per round).  Here a workgroup runs its
// tiles b, b + G, b + 2G, ... (G workgroups, the same tile order as one
// workgroup per tile) with two sets of accumulators: while it computes tile
// r, each K step also stores one of the 18 fragments of tile r - 1, so the
// stores and their arithmetic fill the gaps between MFMAs; only the last
// tile's epilogue stands alone.  The tile loads run on across tiles (the
// last two K steps of a tile issue the next tile's first two stages).
// Stores and loads share vmcnt, which completes in issue order: the wait for
// stage g counts as younger the one stage issued after it and the stores
// of the two K steps since it was issued (4 two-byte stores per q|k
// fragment, 1 eight-byte store per V fragment -- lower bounds on what the
// compiler emits, so the waits are never too lax); compiler barriers keep
// each step's stores after its loads.  Each output element is computed and
// rounded exactly as by gemm_dma_kernel.  Requirements (launch_gemm_dma
// checks): whole tiles (M % 256 == 0, N % 144 == 0), K = 1152 (18 K steps, one
// fragment per step), vcol0 % 144 == 0 (every tile all q|k or all V),
// vectorisable epilogue, at most kPipeTiles tiles per workgroup.
constexpr int kPipeTiles = 6;

__global__ __launch_bounds__(512, 1) void gemm_dma_vt_pipe_kernel(
    const bf16* __restrict__ A, int lda, const bf16* __restrict__ W, int ldw,
    const bf16* __restrict__ bias, int M, int N, Epi epi, int tiles_n, int group_m, int total) {
  constexpr int BM = 256, BN = 144, NW = 8, WM = 32, TM = 2, TN = 9, ST = 3, KT = 18;
  constexpr int ABLK = BM / 8, BBLK = BN / 8, TBLK = ABLK + BBLK, BPW = (TBLK + NW - 1) / NW;
  constexpr int STAGE = (BM + BN) * 64;
  static_assert(TM * TN == KT && KT % ST == 0 && BPW == 7, "one fragment per K step");
  // the stage ring, then 1 KB per tile for its bias row (bf16; the first
  // 288 bytes used)
  __shared__ __attribute__((aligned(1024))) bf16 smem[ST * STAGE + kPipeTiles * 512];
  const bf16* const ebias = smem + ST * STAGE;   // tile r's row at r * 512

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int fr = lane & 15, g = lane >> 4;
  const int G = gridDim.x, b = blockIdx.x;
  const int R = (total - b + G - 1) / G;   // this workgroup's tiles (1 .. kPipeTiles)
  const int tiles_m = M / BM;
  auto tile_of = [&](int r, int& m0, int& n0) {
    const int tile = xcd_remap_dma(b + r * G, total);
    const int per_group = group_m * tiles_n, grp = tile / per_group;
    const int first = grp * group_m, rows_in = min(tiles_m - first, group_m);
    const int in_grp = tile - grp * per_group;
    m0 = (first + in_grp % rows_in) * BM;
    n0 = (in_grp / rows_in) * BN;
  };
  int dst[BPW];
  auto make_src = [&](int m0, int n0, uint32_t (&src)[BPW]) {
#pragma unroll
    for (int i = 0; i < BPW; ++i) {
      int blk = wave + i * NW;
      if (blk >= TBLK) blk -= NW;   // repeat this wave's previous block
      const int lr = (blk < ABLK ? blk : blk - ABLK) * 8 + (lane >> 3);
      const int c = (lane & 7) ^ ((lr >> 1) & 7);
      src[i] = 2u * (uint32_t)(i < ABLK / NW ? (m0 + lr) * lda + c * 8 : (n0 + lr) * ldw + c * 8);
      dst[i] = blk * 1024;
    }
  };
  const __amdgpu_buffer_rsrc_t ra =
      __builtin_amdgcn_make_buffer_rsrc((void*)A, 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rw =
      __builtin_amdgcn_make_buffer_rsrc((void*)W, 0, 0x7fffffff, 0x00020000);
  auto issue = [&](const uint32_t (&src)[BPW], int t, int slot) {
#pragma unroll
    for (int i = 0; i < BPW; ++i)
      dma16<1>(i < ABLK / NW ? ra : rw, (char*)smem + slot * STAGE * 2 + dst[i], src[i], t * 128);
  };

  // every tile's bias row straight into LDS, one direct load per tile from
  // wave 0, before any tile load (so that no wait below has to count them;
  // lanes past the row read neighbouring columns or, past N, zeros)
  if (wave == 0) {
    const __amdgpu_buffer_rsrc_t rb =
        __builtin_amdgcn_make_buffer_rsrc((void*)bias, 0, (uint32_t)N * 2u, 0x00020000);
#pragma unroll
    for (int r = 0; r < kPipeTiles; ++r) {
      if (r >= R) break;
      int m0r, n0r;
      tile_of(r, m0r, n0r);
      dma16<0>(rb, (char*)(ebias + r * 512), 2u * (uint32_t)(n0r + lane * 8), 0);
    }
  }

  int m0, n0, m0n = 0, n0n = 0;
  uint32_t src_c[BPW], src_n[BPW];
  tile_of(0, m0, n0);
  make_src(m0, n0, src_c);
  if (R > 1) tile_of(1, m0n, n0n);
#pragma unroll
  for (int s = 0; s < ST - 1; ++s) issue(src_c, s, s);

  f32x4 acc[TM][TN];
  bf16x4 prev[TM][TN];   // the previous tile's outputs, rounded, waiting to be stored
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto frag = [&](const bf16* base, int row, int c) {
    return *(const bf16x8*)((const char*)base + row * 128 + ((c ^ ((row >> 1) & 7)) << 4));
  };
  auto compute = [&](int slot) {
    const bf16* sA = smem + slot * STAGE;
    const bf16* sB = sA + BM * 64;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      bf16x8 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) af[i] = frag(sA, wave * WM + i * 16 + fr, kk * 4 + g);
#pragma unroll
      for (int j = 0; j < TN; ++j) bfr[j] = frag(sB, j * 16 + fr, kk * 4 + g);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
  };
  // fragment (i, j) of a finished tile at (tm0, tn0) with bias row r, rounded
  // exactly as the whole-tile epilogues of gemm_dma_kernel round it: V
  // columns acc + b, q|k columns (acc + b) * qscale for the query columns
  auto round_frag = [&](int i, int j, int tn0, bool is_v, int r) {
    const int n = tn0 + j * 16 + fr;
    const float bv = (float)ebias[r * 512 + j * 16 + fr];
    const float qs = !is_v && n < epi.qcols ? epi.qscale : 1.f;
    bf16x4 w;
#pragma unroll
    for (int rr = 0; rr < 4; ++rr)
      w[rr] = is_v ? (bf16)(acc[i][j][rr] + bv) : (bf16)((acc[i][j][rr] + bv) * qs);
    return w;
  };
  // its stores: V^T four tokens per store, q|k one element per store
  auto store_frag = [&](bf16x4 w, int i, int j, int tm0, int tn0, bool is_v) {
    const int n = tn0 + j * 16 + fr, mb = tm0 + wave * WM + i * 16 + g * 4;
    if (is_v) {
      *(bf16x4*)(epi.vt + (size_t)(n - epi.vcol0) * epi.ldvt + mb) = w;
    } else {
      bf16* o = (bf16*)epi.out + n;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) o[(size_t)(mb + rr) * epi.ldo] = w[rr];
    }
  };

  bool cur_v = n0 >= epi.vcol0, prev_v = false;
  int pm0 = 0, pn0 = 0;
  int e_last = 0;   // stores per K step during the previous tile
  for (int r = 0; r < R; ++r) {
    const int e_cur = r > 0 ? (prev_v ? 1 : 4) : 0;   // stores per K step during this tile
    const bool next = r + 1 < R;
#pragma unroll
    for (int t = 0; t < KT; ++t) {
      // younger than stage (r, t): the stores of the two steps since it was
      // issued and the stage issued one step after it (if any)
      const int e2 = t >= 2 ? e_cur : e_last, e1 = t >= 1 ? e_cur : e_last;
      const bool younger_stage = t + 1 < KT || next;
      wait_vmcnt_dyn15(e2 + e1 + (younger_stage ? BPW : 0));
      block_barrier();
      if (t + ST - 1 < KT) {
        issue(src_c, t + ST - 1, (t + ST - 1) % ST);
      } else if (next) {
        make_src(m0n, n0n, src_n);
        issue(src_n, t + ST - 1 - KT, (t + ST - 1) % ST);
      }
      asm volatile("" ::: "memory");   // this step's stores stay after its loads
      compute(t % ST);
      if (r > 0) store_frag(prev[t / TN][t % TN], t / TN, t % TN, pm0, pn0, prev_v);
      asm volatile("" ::: "memory");   // ... and before the next step's wait
    }
    if (next) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          prev[i][j] = round_frag(i, j, n0, cur_v, r);
          acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
      prev_v = cur_v;
      pm0 = m0;
      pn0 = n0;
      m0 = m0n;
      n0 = n0n;
      cur_v = n0 >= epi.vcol0;
      make_src(m0, n0, src_c);
      if (r + 2 < R) tile_of(r + 2, m0n, n0n);
      e_last = e_cur;
    } else {
      // the last tile's epilogue
#pragma unroll
      for (int f = 0; f < TM * TN; ++f)
        store_frag(round_frag(f / TN, f % TN, n0, cur_v, r), f / TN, f % TN, m0, n0, cur_v);
    }
  }
}

template <int BM, int BN, int WGM, int WGN, int ST, int AUX>
hipError_t gemm_dma_dispatch(const bf16* A, int lda, const bf16* W, int ldw, const bf16* bias,
                             int M, int N, int K, int kind, const Epi& epi, int vec_ok,
                             int group_m, hipStream_t st) {
  const int tn = (N + BN - 1) / BN, tm = (M + BM - 1) / BM;
  dim3 grid(tm * tn), block(64 * WGM * WGN);
#define T2I_DMA_CASE(K_)                                                                      \
  case K_:                                                                                    \
    hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WGM, WGN, ST, K_, AUX, XNone>), grid, block, 0, st, \
                       A, lda, W, ldw, bias, M, N, K, epi, tn, group_m, vec_ok, XNone{});     \
    break;
  switch (kind) {
    T2I_DMA_CASE(EPI_STORE)
    T2I_DMA_CASE(EPI_GELU)
    T2I_DMA_CASE(EPI_RESID)
    T2I_DMA_CASE(EPI_RESID_GATED)
    T2I_DMA_CASE(EPI_SPLIT_VT)
    T2I_DMA_CASE(EPI_STORE_F32)
    default: return hipErrorInvalidValue;
  }
#undef T2I_DMA_CASE
  return hipGetLastError();
}

// Large-M projections (tile shapes and orders measured on MI355X at the DiT's
// and the joint-attention model's shapes).  Operand loads that miss the XCD's
// L2 bound these GEMMs: a CU takes 30-57 bytes per clock of direct loads from
// L2 but only 10-13 from the memory-side cache or HBM, and in these GEMMs it
// averages ~17.  Bytes per FLOP -- (BM + BN) / (BM BN) -- and the L2 reuse of
// the tile order decide, together with filling whole rounds of 256
// workgroups:
//   256 x 288 (8 waves of 64 x 144) where N is a multiple of 288 and its
//             rounds cost less (fc1: N = 4608, M = 8192 -> 512 tiles);
//   256 x 256 for long K where N is a multiple of 256 with whole rounds
//             (joint-attention MLP up-projection: N = 12288 -> 768 tiles);
//   256 x 144 (8 waves of 32 x 144, three stages) for the other DiT widths;
//   256 x 192 (8 waves of 64 x 96) where that fills whole rounds (N = 3072);
//   256 x 128 otherwise.
// Row blocks per tile group (see gemm_dma_kernel): 8 for long K, 2 for the
// 288-wide tiles at short K, 1 for the 144-wide residual updates.  All load
// with cache policy bit 0 (sc0) set, which measured faster.
// Projections of a few hundred to ~2000 rows (the 512-px DiT's 1024, the
// single small requests of a packed batch) on narrower tiles with deeper
// rings: there the register-staged kernel waits a load latency per K step.
// Row height 128, 64 or 32: one workgroup per CU (the rings take most of the
// LDS), so a launch costs about (rounds of 256 tiles) x (the tile's bytes per
// K step, proportional to BM + 144); the smallest estimate wins, ties to the
// taller tile (1024 rows: 32 x 144 for the 1152-wide layers -> 256 tiles,
// 128 x 144 for qkv and fc1).  Every output element accumulates the same
// MFMAs in the same K order as in every other GEMM path, so results do not
// depend on the choice.
hipError_t launch_gemm_dma_small(const bf16* A, int lda, const bf16* W, int ldw, const bf16* bias,
                                 int M, int N, int K, int kind, const Epi& epi, int vec_ok,
                                 hipStream_t st) {
  const long tn = N / 144;
  auto cost = [&](int bm) { return ((((M + bm - 1) / bm) * tn + 255) / 256) * (bm + 144); };
  const long c128 = cost(128), c64 = cost(64), c32 = cost(32);
  if (c128 <= c64 && c128 <= c32)
    return gemm_dma_dispatch<128, 144, 8, 1, 4, 1>(A, lda, W, ldw, bias, M, N, K, kind, epi, vec_ok,
                                                   8, st);
  if (c64 <= c32)
    return gemm_dma_dispatch<64, 144, 4, 1, 5, 1>(A, lda, W, ldw, bias, M, N, K, kind, epi, vec_ok,
                                                  8, st);
  return gemm_dma_dispatch<32, 144, 2, 1, 6, 1>(A, lda, W, ldw, bias, M, N, K, kind, epi, vec_ok,
                                                16, st);
}

hipError_t launch_gemm_dma(const bf16* A, int lda, const bf16* W, int ldw, const bf16* bias,
                           int M, int N, int K, int kind, const Epi& epi, int vec_ok,
                           hipStream_t st) {
  const long mt = (M + 255) / 256;
  const bool longk = K >= 2048;
  // 288 wide where its rounds cost less: a round of 256 x 288 tiles takes
  // ~1.8x a round of 256 x 144 tiles (measured at 8192 rows), so the wider
  // tile wins when it needs fewer than 5/9 of the rounds (fc1 at 8192 rows:
  // 2 rounds against 4; the 1152-wide layers at 12 032 rows: 1 against 2)
  if (N % 288 == 0) {
    const long r288 = (mt * (N / 288) + 255) / 256, r144 = (mt * (N / 144) + 255) / 256;
    if (r288 * 9 <= r144 * 5)
      return gemm_dma_dispatch<256, 288, 4, 2, 2, 1>(A, lda, W, ldw, bias, M, N, K, kind, epi,
                                                     vec_ok, longk ? 8 : 2, st);
  }
  if (longk && N % 256 == 0 && (mt * (N / 256)) % 256 == 0)
    return gemm_dma_dispatch<256, 256, 4, 2, 2, 1>(A, lda, W, ldw, bias, M, N, K, kind, epi, vec_ok,
                                                   8, st);
  if (N % 144 == 0) {
    const int gm = longk ? 8 : (kind == EPI_RESID || kind == EPI_RESID_GATED) ? 1 : 8;
    const long tiles = mt * (N / 144);
    if (kind == EPI_SPLIT_VT && vec_ok && M % 256 == 0 && K == 18 * 64 && epi.vcol0 % 144 == 0 &&
        tiles > 256 && tiles <= (long)kPipeTiles * 256) {
      hipLaunchKernelGGL(gemm_dma_vt_pipe_kernel, dim3(256), dim3(512), 0, st, A, lda, W, ldw, bias,
                         M, N, epi, N / 144, gm, (int)tiles);
      return hipGetLastError();
    }
    return gemm_dma_dispatch<256, 144, 8, 1, 3, 1>(A, lda, W, ldw, bias, M, N, K, kind, epi, vec_ok,
                                                   gm, st);
  }
  if (N % 192 == 0 && (mt * (N / 192)) % 256 == 0)
    return gemm_dma_dispatch<256, 192, 4, 2, 2, 1>(A, lda, W, ldw, bias, M, N, K, kind, epi, vec_ok,
                                                   8, st);
  return gemm_dma_dispatch<256, 128, 4, 2, 3, 1>(A, lda, W, ldw, bias, M, N, K, kind, epi, vec_ok, 8,
                                                 st);
}

// The cross-attention query projection with the cross-attention fused in
// (gemm_dma_kernel with XAttnArgs), where the shapes fit it: head dimension
// 72 (a 144-wide tile holds two heads), K a multiple of 3 x 64 (the text
// tiles load during the last K step), every sequence's query rows a whole
// number of 256-row tiles, texts of 1 .. 128 keys within V^T's row length,
// 16-byte aligned operands.  Otherwise
// hipErrorNotSupported, launching nothing: the caller then runs the
// projection and attn_cross_kernel separately, which give the same bits.
// check_only: the checks alone (hipSuccess where the fused kernel applies).
hipError_t launch_gemm_xattn(const bf16* A, int lda, const bf16* W, int ldw, const bf16* bias,
                             int M, int N, int K, const Epi& epi, int heads, int head_dim,
                             const XAttnArgs& xa, hipStream_t st, bool check_only) {
  auto al = [](const void* p, int a) { return ((uintptr_t)p % a) == 0; };
  if (head_dim != 72 || N != heads * 72 || N % 144 || M < 256 || M % 256 || K < 192 || K % 192 ||
      lda % 8 || ldw % 8 || !al(A, 16) || !al(W, 16) || !al(bias, 8) || !al(xa.O, 16) ||
      !al(xa.K, 16) || !al(xa.Vt, 16) || xa.ldo % 8 || xa.ldo < N || xa.ldk < N || xa.ldk % 8 ||
      xa.ldvt % 8 || xa.n < 1 || xa.n > kMaxSeq)
    return hipErrorNotSupported;
  if ((size_t)2 * M * lda >= 0x7fffffff || (size_t)2 * N * ldw >= 0x7fffffff)
    return hipErrorNotSupported;
  int next = 0, k_rows = 0;
  for (int s = 0; s < xa.n; ++s) {
    if (xa.q_start[s] != next || xa.q_len[s] <= 0 || xa.q_len[s] % 256 || xa.k_len[s] < 1 ||
        xa.k_len[s] > 128 || xa.k_start[s] < 0 || xa.k_start[s] % 8 ||
        xa.k_start[s] + xa.k_len[s] > xa.ldvt)
      return hipErrorNotSupported;
    next += xa.q_len[s];
    k_rows = std::max(k_rows, xa.k_start[s] + xa.k_len[s]);
  }
  if (next != M) return hipErrorNotSupported;
  // text tile loads address K and V^T with byte offsets below 2^31
  if ((size_t)2 * heads * head_dim * xa.ldvt > 0x7fffffff ||
      (size_t)2 * (k_rows + 64) * xa.ldk > 0x7fffffff)
    return hipErrorNotSupported;
  if (check_only) return hipSuccess;
  const int tn = N / 144, tm = M / 256;
  hipLaunchKernelGGL((gemm_dma_kernel<256, 144, 8, 1, 3, EPI_STORE, 1, XAttnArgs>), dim3(tm * tn),
                     dim3(512), 0, st, A, lda, W, ldw, bias, M, N, K, epi, tn, 8, 1, xa);
  return hipGetLastError();
}

// Counter calibration: read `chunks` KB of src once through the same direct
// HBM -> LDS path (buffer_load_dwordx4 ... lds, 1 KB per wave instruction) the
// GEMM and attention kernels use, writing nothing to global memory but one
// float per workgroup.  Waves never wait inside the loop (the hardware stalls
// issue once its outstanding-load counter is full), so the loads stream.
__global__ __launch_bounds__(256) void dma_read_kernel(const char* __restrict__ src, int chunks,
                                                       float* __restrict__ sink) {
  __shared__ __attribute__((aligned(1024))) char smem[4 * 1024];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const __amdgpu_buffer_rsrc_t r =
      __builtin_amdgcn_make_buffer_rsrc((void*)src, 0, 0x7fffffff, 0x00020000);
  const int nw = gridDim.x * 4;
  for (int c = blockIdx.x * 4 + wave; c < chunks; c += nw)
    dma16<0>(r, smem + wave * 1024, (uint32_t)c * 1024u + (uint32_t)lane * 16u, 0);
  wait_vmcnt<0>();
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = *(const float*)smem;
}

hipError_t launch_dma_read(const void* src, size_t bytes, float* sink, hipStream_t st) {
  if (bytes == 0) return hipSuccess;
  if (bytes % 1024 || bytes > ((size_t)1 << 31) - 1024) return hipErrorInvalidValue;
  hipLaunchKernelGGL(dma_read_kernel, dim3(kDmaReadGroups), dim3(256), 0, st, (const char*)src,
                     (int)(bytes / 1024), sink);
  return hipGetLastError();
}

}  // namespace t2i
