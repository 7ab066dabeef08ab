// Multi-head attention over packed variable-length sequences (self-attention,
// cross-attention to text, joint attention) on gfx950.
//
// attn_bf16_kernel: flash-style, one workgroup = 4 waves = 128 queries of one
// head of one sequence; each wave owns 32 queries (two 16-query MFMA tiles).
// Keys/values stream through LDS 64 at a time.  Everything is arranged so that
// a lane always holds data of ONE query:
//   * scores are computed transposed, S^T = K Q^T, with v_mfma_f32_16x16x32_bf16
//     (A = K fragment, B = Q fragment kept in registers for the whole loop):
//     the C fragment gives lane l the scores of query (l & 15) against keys
//     4*(l >> 4) + 0..3 of each 16-key tile;
//   * the output is accumulated transposed, O^T = V^T P^T: the B operand is
//     exactly the lane's own probabilities (8 keys of two adjacent 16-key
//     tiles), the A operand is read from a V^T tile in LDS, and the C fragment
//     again gives lane l query (l & 15) -- so the online-softmax rescale of the
//     output needs no data exchange between lanes.
// The row max needs two cross-lane steps per tile (the 4 lanes of a query);
// the row sums ride on a ones row of V^T where the head dimension has padding
// (else they are kept per lane and combined once at the end).  The head
// dimension is padded with zeros to a multiple of 32 for Q K^T and to a
// multiple of 16 for P V (72 -> 96 / 80); the padding never reaches memory.
//
// attn_f32_kernel: plain fp32 online softmax, one thread per query, for the
// fp32 model.
#include "t2i_internal.h"

namespace t2i {

__device__ __forceinline__ int xcd_remap_attn(int b, int nb) {
  const int q = nb >> 3, r = nb & 7;
  const int x = b & 7, j = b >> 3;
  return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + j;
}

// Position of tile key k (0..63) in a staged V^T row.  Within each 32-key
// chunk the keys a lane multiplies -- 4g..4g+3 and 16+4g..16+4g+3, the
// probabilities its S^T fragment holds -- are stored next to each other at
// 8g..8g+7, so one conflict-free 16-byte LDS read feeds the PV MFMA.
__device__ __forceinline__ int vpos(int k) {
  const int kk = k & 31;
  return (k & 32) + 8 * ((kk & 15) >> 2) + 4 * (kk >> 4) + (kk & 3);
}

// Flattened tile -> (head, sequence, query tile).  Tiles of one head and one
// sequence are consecutive so that they land on one XCD and share K/V in L2.
__device__ __forceinline__ void decode_tile(const AttnMap& m, int heads, int L, int& h, int& s,
                                            int& j) {
  const int total = m.tile_start[m.n];
  h = L / total;
  const int t = L - h * total;
  s = 0;
#pragma unroll 1
  for (int i = 1; i < m.n; ++i) s += (t >= m.tile_start[i]) ? 1 : 0;
  j = t - m.tile_start[s];
}

template <int HD, int QT>
__global__ __launch_bounds__(256, 2) void attn_bf16_kernel(AttnMap map, int heads,
                                                           const bf16* __restrict__ Q, int ldq,
                                                           const bf16* __restrict__ K, int ldk,
                                                           const bf16* __restrict__ Vt, int ldvt,
                                                           bf16* __restrict__ O, int ldo,
                                                           float scale_log2) {
  constexpr int BQ = 4 * QT * 16, BKV = 64;
  constexpr int DC = (HD + 31) / 32;   // 32-wide chunks of d for Q K^T
  constexpr int HDP = DC * 32;
  constexpr int DT = (HD + 15) / 16;   // 16-wide tiles of d for P V
  constexpr int HDO = DT * 16;
  // row sums: a spare V^T row of ones where the head dimension has padding,
  // else one more P V MFMA against a ones fragment held in registers
  constexpr bool ONES = HD < HDO;
  constexpr int VP = BKV + 8;          // LDS pitch of a V^T row (bf16)
  constexpr int CPR = HD / 8;          // 16-byte chunks per K row
  // K tile, chunk-major: block b (1 KB) holds d = 8b .. 8b+7 of the 64 keys,
  // key k at byte 16k; block CPR is all zeros (the d padding of Q K^T)
  constexpr int KBLK = CPR + 1;
  constexpr int KST = KBLK * 512;      // bf16 elements per K stage
  constexpr int KBPW = (CPR + 3) / 4;  // K load instructions per wave
  constexpr int VCH = HD * (BKV / 8);
  constexpr int VPT = (VCH + 255) / 256;
  __shared__ __attribute__((aligned(1024))) bf16 Ks[2][KST];
  __shared__ bf16 Vs[2][HDO * VP];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int h, s, j;
  decode_tile(map, heads, xcd_remap_attn(blockIdx.x, gridDim.x), h, s, j);
  const int q_beg = map.q_start[s], q_end = q_beg + map.q_len[s];
  // key tiles: those of segment 1, then those of segment 2
  const int k1 = map.k_start[s], n1 = map.k_len[s];
  const int k2 = map.k2_start[s], n2 = map.k2_len[s];
  const int t1 = (n1 + BKV - 1) / BKV, nt = t1 + (n2 + BKV - 1) / BKV;
  auto tile_keys = [&](int ti, int& kv0, int& kend) {
    if (ti < t1) {
      kv0 = k1 + ti * BKV;
      kend = k1 + n1;
    } else {
      kv0 = k2 + (ti - t1) * BKV;
      kend = k2 + n2;
    }
  };
  const int qrow0 = q_beg + j * BQ + wave * (QT * 16);
  const int g = lane >> 4, fr = lane & 15;

  // zero both buffers once: the K zero block and the V^T padding rows stay zero
  for (int i = tid; i < 2 * KST; i += 256) (&Ks[0][0])[i] = (bf16)0.f;
  for (int i = tid; i < 2 * HDO * VP; i += 256) (&Vs[0][0])[i] = (bf16)0.f;

  // K tiles move HBM -> LDS directly (global_load_lds_dwordx4): instruction
  // for block b has lane = key and fetches that key's d-chunk b.  Waves with
  // fewer blocks repeat one (identical bytes).  Key rows past the sequence are
  // clamped to its last key; their scores are masked.
  int kblk[KBPW];
#pragma unroll
  for (int i = 0; i < KBPW; ++i) kblk[i] = min(wave + 4 * i, CPR - 1);
  auto kload = [&](int kv0, int k_end, int buf) {
    const int gk = min(kv0 + lane, k_end - 1);
    const bf16* src = K + (size_t)gk * ldk + h * HD;
#pragma unroll
    for (int i = 0; i < KBPW; ++i)
      __builtin_amdgcn_global_load_lds(
          (__attribute__((address_space(1))) void*)(src + kblk[i] * 8),
          (__attribute__((address_space(3))) void*)(&Ks[buf][kblk[i] * 512]), 16, 0, 0);
  };

  bf16x8 vr[VPT];
  auto gload = [&](int kv0, int k_end) {
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int c = tid + 256 * i;
      vr[i] = bf16x8{};
      if (c < VCH) {
        const int d = c >> 3, gk = kv0 + (c & 7) * 8;
        if (gk < k_end) {
          vr[i] = *(const bf16x8*)(Vt + (size_t)(h * HD + d) * ldvt + gk);
          if (gk + 8 > k_end) {
#pragma unroll
            for (int e = 0; e < 8; ++e)
              if (gk + e >= k_end) vr[i][e] = (bf16)0.f;
          }
        }
      }
    }
  };
  auto sstore = [&](int buf, int kv0, int k_end) {
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int c = tid + 256 * i;
      if (c < VCH) {
        // keys 8(c&7) .. +7 of row c>>3: two groups of four, each to its
        // permuted position (see vpos)
        bf16* row = &Vs[buf][(c >> 3) * VP];
        const int k = (c & 7) * 8;
        *(bf16x4*)&row[vpos(k)] = bf16x4{vr[i][0], vr[i][1], vr[i][2], vr[i][3]};
        *(bf16x4*)&row[vpos(k + 4)] = bf16x4{vr[i][4], vr[i][5], vr[i][6], vr[i][7]};
      }
    }
    if (ONES && tid < BKV) Vs[buf][HD * VP + vpos(tid)] = (bf16)(kv0 + tid < k_end ? 1.f : 0.f);
  };

  // Q fragments (B operand of S^T): query qrow0 + qt*16 + fr, d = c*32 + g*8 .. +7,
  // pre-multiplied by log2(e)/sqrt(d) so that scores come out in log2 units
  bf16x8 qf[QT][DC];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int qr = qrow0 + qt * 16 + fr;
#pragma unroll
    for (int c = 0; c < DC; ++c) {
      const int d = c * 32 + g * 8;
      qf[qt][c] = bf16x8{};
      if (qr < q_end && d < HD) {
        const bf16x8 raw = *(const bf16x8*)(Q + (size_t)qr * ldq + h * HD + d);
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[qt][c][e] = (bf16)((float)raw[e] * scale_log2);
      }
    }
  }

  // Online softmax with a lazily updated maximum: every score accumulator
  // starts at -m_run (the MFMA's C operand), so S' = s - m_run arrives ready
  // for exp2.  While no S' exceeds 8 the stale maximum is kept: probabilities
  // stay <= 256 and the common scale cancels between numerator and row sum.
  f32x4 o[QT][DT], osum[QT];
  float m_run[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    m_run[qt] = -INFINITY;
    osum[qt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[qt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // A fragment of a [16 x 32] tile whose row 0 is all ones (lane fr == 0)
  bf16x8 ones_frag;
#pragma unroll
  for (int e = 0; e < 8; ++e) ones_frag[e] = (bf16)(fr == 0 ? 1.f : 0.f);

  // K fragment of 32-wide d chunk c: block 4c + g (the zero block past HD)
  int koff[DC];
#pragma unroll
  for (int c = 0; c < DC; ++c) koff[c] = min(4 * c + g, CPR) * 512 + fr * 8;

  __syncthreads();          // zero-fill done before the first tile lands
  {
    int kv0, kend;
    tile_keys(0, kv0, kend);
    kload(kv0, kend, 0);
    gload(kv0, kend);
    sstore(0, kv0, kend);
  }
  __syncthreads();          // (waits for the K loads too)
  int buf = 0;
  for (int ti = 0; ti < nt; ++ti) {
    int kv0, k_end, nkv0 = 0, nkend = 0;
    tile_keys(ti, kv0, k_end);
    const bool next = ti + 1 < nt;
    if (next) {
      tile_keys(ti + 1, nkv0, nkend);
      kload(nkv0, nkend, buf ^ 1);
      gload(nkv0, nkend);
    }
    const bool ragged = kv0 + BKV > k_end;
    const bf16* Kb = Ks[buf];
    const bf16* Vb = Vs[buf];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      // re-read the K / V^T fragments for every query tile instead of keeping
      // all of them live across tiles (register pressure, not LDS traffic,
      // limits this kernel)
      asm volatile("" ::: "memory");
      // d-chunk outer, key tile inner: four independent accumulation chains,
      // each started from -m_run
      const float negm = m_run[qt] == -INFINITY ? 0.f : -m_run[qt];
      const f32x4 cinit = f32x4{negm, negm, negm, negm};
      f32x4 sc[4];
#pragma unroll
      for (int c = 0; c < DC; ++c) {
        bf16x8 kf[4];
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) kf[kt] = *(const bf16x8*)&Kb[koff[c] + kt * 128];
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
          sc[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[kt], qf[qt][c],
                                                           c == 0 ? cinit : sc[kt], 0, 0, 0);
      }
      if (ragged) {
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (kv0 + kt * 16 + g * 4 + r >= k_end) sc[kt][r] = -INFINITY;
      }
      float lm = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
        lm = fmaxf(fmaxf(lm, fmaxf(sc[kt][0], sc[kt][1])), fmaxf(sc[kt][2], sc[kt][3]));
      if (ti == 0 || __any(lm > 8.0f)) {
        // new maximum: the query's 64 scores sit in the 4 lanes fr, fr+16, ..
        float mx = fmaxf(lm, __shfl_xor(lm, 16, 64));
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        const float m_new = fmaxf(m_run[qt], mx - negm);
        const float delta = m_new + negm;          // shift of the subtracted value
        const float alpha = __builtin_amdgcn_exp2f(m_run[qt] - m_new);
        m_run[qt] = m_new;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) sc[kt][r] -= delta;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[qt][dt] *= alpha;
        osum[qt] *= alpha;
      }
      bf16x8 pf[2];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          pf[kt >> 1][(kt & 1) * 4 + r] = (bf16)__builtin_amdgcn_exp2f(sc[kt][r]);
      // key chunk outer, d tile inner: DT independent accumulation chains.
      // The lane's 8 keys are contiguous in the permuted V^T row: one 16-byte read.
#pragma unroll
      for (int kc = 0; kc < 2; ++kc) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const bf16x8 vf = *(const bf16x8*)&Vb[(dt * 16 + fr) * VP + kc * 32 + g * 8];
          o[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[kc], o[qt][dt], 0, 0, 0);
        }
        if (!ONES)
          osum[qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones_frag, pf[kc], osum[qt], 0, 0, 0);
      }
    }
    if (next) sstore(buf ^ 1, nkv0, nkend);
    __syncthreads();
    buf ^= 1;
  }

#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    float l;
    if (ONES) {
      // row HD of O^T = sum of the probabilities: tile HD/16, row HD%16, held
      // by the lanes with g = (HD%16)/4 as component (HD%16)%4
      constexpr int LT = HD / 16, LR = HD % 16;
      l = __shfl(o[qt][LT][LR % 4], (LR / 4) * 16 + fr, 64);
    } else {
      l = __shfl(osum[qt][0], fr, 64);   // row 0 of the ones product
    }
    const float inv = 1.0f / l;
    const int qr = qrow0 + qt * 16 + fr;
    if (qr >= q_end) continue;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const int d = dt * 16 + g * 4;
      if (d < HD) {
        bf16x4 w;
#pragma unroll
        for (int r = 0; r < 4; ++r) w[r] = (bf16)(o[qt][dt][r] * inv);
        *(bf16x4*)(O + (size_t)qr * ldo + h * HD + d) = w;
      }
    }
  }
}

// ---------------------------------------------------------------------------

template <int HD>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnMap map, int heads,
                                                      const float* __restrict__ Q, int ldq,
                                                      const float* __restrict__ K, int ldk,
                                                      const float* __restrict__ V, int ldv,
                                                      float* __restrict__ O, int ldo, float scale) {
  constexpr int BQ = 64, BKV = 32;
  __shared__ float Ks[BKV][HD];
  __shared__ float Vs[BKV][HD];
  int h, s, j;
  decode_tile(map, heads, blockIdx.x, h, s, j);
  const int q_beg = map.q_start[s], q_end = q_beg + map.q_len[s];
  const int qr = q_beg + j * BQ + threadIdx.x;
  const bool active = qr < q_end;
  float q[HD], acc[HD];
#pragma unroll
  for (int d = 0; d < HD; ++d) {
    q[d] = active ? Q[(size_t)qr * ldq + h * HD + d] : 0.f;
    acc[d] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int seg = 0; seg < 2; ++seg) {
    const int k_beg = seg ? map.k2_start[s] : map.k_start[s];
    const int k_end = k_beg + (seg ? map.k2_len[s] : map.k_len[s]);
    for (int kv0 = k_beg; kv0 < k_end; kv0 += BKV) {
      __syncthreads();
      for (int i = threadIdx.x; i < BKV * HD; i += 64) {
        const int key = i / HD, d = i - key * HD, gk = kv0 + key;
        Ks[key][d] = gk < k_end ? K[(size_t)gk * ldk + h * HD + d] : 0.f;
        Vs[key][d] = gk < k_end ? V[(size_t)gk * ldv + h * HD + d] : 0.f;
      }
      __syncthreads();
      const int nk = min(BKV, k_end - kv0);
      for (int key = 0; key < nk; ++key) {
        float sdot = 0.f;
#pragma unroll
        for (int d = 0; d < HD; ++d) sdot = fmaf(q[d], Ks[key][d], sdot);
        sdot *= scale;
        const float m_new = fmaxf(m, sdot);
        const float corr = expf(m - m_new);
        const float p = expf(sdot - m_new);
        l = l * corr + p;
#pragma unroll
        for (int d = 0; d < HD; ++d) acc[d] = acc[d] * corr + p * Vs[key][d];
        m = m_new;
      }
    }
  }
  if (active) {
    const float inv = 1.0f / l;
#pragma unroll
    for (int d = 0; d < HD; ++d) O[(size_t)qr * ldo + h * HD + d] = acc[d] * inv;
  }
}

// 16-query tiles per wave: 4 (64 queries) while the output accumulators fit
// next to everything else in 256 registers, 2 for the widest heads
constexpr int query_tiles(int hd) { return hd > 96 ? 2 : 4; }
int attention_query_tile(bool bf16_io, int head_dim) {
  if (!bf16_io) return 64;
  return 4 * 16 * (head_dim > 96 ? 2 : 4);
}

template <int HD>
static hipError_t launch_hd(bool bf16_io, int heads, const AttnMap& map, const void* q, int ldq,
                            const void* k, int ldk, const void* v, int ldv, void* o, int ldo,
                            hipStream_t st) {
  const int tiles = map.tile_start[map.n] * heads;
  if (tiles == 0) return hipSuccess;
  if (bf16_io) {
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)HD);
    hipLaunchKernelGGL((attn_bf16_kernel<HD, query_tiles(HD)>), dim3(tiles), dim3(256), 0, st, map, heads,
                       (const bf16*)q, ldq, (const bf16*)k, ldk, (const bf16*)v, ldv, (bf16*)o, ldo,
                       scale_log2);
  } else {
    const float scale = 1.0f / sqrtf((float)HD);
    hipLaunchKernelGGL(attn_f32_kernel<HD>, dim3(tiles), dim3(64), 0, st, map, heads,
                       (const float*)q, ldq, (const float*)k, ldk, (const float*)v, ldv, (float*)o,
                       ldo, scale);
  }
  return hipGetLastError();
}

hipError_t launch_attention(bool bf16_io, int heads, int head_dim, const AttnMap& map,
                            const void* q, int ldq, const void* k, int ldk, const void* v, int ldv,
                            void* o, int ldo, hipStream_t st) {
  switch (head_dim) {
    case 8: return launch_hd<8>(bf16_io, heads, map, q, ldq, k, ldk, v, ldv, o, ldo, st);
    case 32: return launch_hd<32>(bf16_io, heads, map, q, ldq, k, ldk, v, ldv, o, ldo, st);
    case 64: return launch_hd<64>(bf16_io, heads, map, q, ldq, k, ldk, v, ldv, o, ldo, st);
    case 72: return launch_hd<72>(bf16_io, heads, map, q, ldq, k, ldk, v, ldv, o, ldo, st);
    case 128: return launch_hd<128>(bf16_io, heads, map, q, ldq, k, ldk, v, ldv, o, ldo, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace t2i
