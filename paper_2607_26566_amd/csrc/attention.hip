// Multi-head attention over packed variable-length sequences (self-attention,
// cross-attention to text, joint attention) on gfx950.
//
// attn_bf16_kernel: flash-style, one workgroup = 8 waves = 256 queries of one
// head of one sequence; each wave owns 32 queries.  Keys and values stream
// through an LDS ring, 64 keys per tile, filled by direct HBM->LDS buffer
// loads that four of the waves issue several tiles ahead (5 stages and one
// barrier per two tiles up to head dimension 72; 4 stages above; 3 stages in
// the 2- and 4-wave workgroups of small launches and cross-attention).
// Everything is arranged so that a lane always holds data of ONE query:
//   * scores are computed transposed, S^T = K Q^T, with
//     v_mfma_f32_32x32x16_bf16 (A = K fragment from LDS, B = the query's Q
//     fragment, kept in registers for the whole loop): lane l gets query
//     (l & 31) against 16 keys of each 32-key block;
//   * the output is accumulated transposed, O^T = V^T P^T: the B operand is
//     exactly the lane's own probabilities, the A operand a V^T fragment from
//     LDS, and the C fragment again belongs to query (l & 31) -- so the
//     online-softmax rescale of the output needs no data exchange between
//     lanes;
//   * the softmax shift rides in a spare slot of the Q K^T contraction (Q
//     carries -m, K a 1), so scores leave the MFMA as s - m; the maximum is
//     updated lazily (only when a score exceeds it by 2^8);
//   * row sums come from a ones row of V^T where the head dimension has
//     padding (72 -> 96), else from a per-lane sum combined once at the end;
//   * the next tile's scores are issued before this tile's exponentials, so
//     the two overlap -- up to head dimension 72 in a fixed slot order that
//     spreads the exponentials over the MFMAs.
//
// attn_f32_kernel: plain fp32 online softmax, one thread per query, for the
// fp32 model.
#include <algorithm>

#include "t2i_internal.h"
#include "xattn_tile.h"

namespace t2i {

// Word 3 of a raw buffer resource on gfx950: 32-bit data format, no swizzle;
// offsets are bytes and reads at or past the extent return zero.
constexpr int kBufWord3 = 0x00020000;

__device__ __forceinline__ int xcd_remap_attn(int b, int nb) {
  const int q = nb >> 3, r = nb & 7;
  const int x = b & 7, j = b >> 3;
  return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + j;
}

// s_waitcnt vmcnt(N), lgkmcnt / expcnt untouched
// (vmcnt is 6 bits: bits 3..0 and 15..14 of the immediate)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// s_waitcnt vmcnt(n) for a wave-uniform n < 32 known only at run time
// (larger n wait for vmcnt(31), which is stricter).
__device__ __forceinline__ void wait_vmcnt_dyn(int n) {
  switch (n) {
#define T2I_W(N_) case N_: wait_vmcnt<N_>(); break;
    T2I_W(0) T2I_W(1) T2I_W(2) T2I_W(3) T2I_W(4) T2I_W(5) T2I_W(6) T2I_W(7)
    T2I_W(8) T2I_W(9) T2I_W(10) T2I_W(11) T2I_W(12) T2I_W(13) T2I_W(14) T2I_W(15)
    T2I_W(16) T2I_W(17) T2I_W(18) T2I_W(19) T2I_W(20) T2I_W(21) T2I_W(22) T2I_W(23)
    T2I_W(24) T2I_W(25) T2I_W(26) T2I_W(27) T2I_W(28) T2I_W(29) T2I_W(30)
#undef T2I_W
    default: wait_vmcnt<31>(); break;
  }
}

__device__ __forceinline__ void attn_barrier() {
  // this wave's LDS accesses are complete, then s_barrier (no wait for
  // outstanding global loads, which __syncthreads would add).  The wait is
  // the builtin so that the compiler's wait-count tracking sees it: after it
  // no scalar load can be pending, and the waits for LDS fragment reads
  // further on can then count reads instead of draining them all.
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0), vmcnt / expcnt untouched
  asm volatile("s_barrier" ::: "memory");
}

// Flattened tile -> (head, sequence, query tile).  HEAD_MINOR = false: tiles
// of one head and one sequence are consecutive so that they land on one XCD
// and share K/V in L2.  HEAD_MINOR = true (cross-attention, whose K/V for all
// heads fit in L2): the heads of one query tile are consecutive, so the
// 128-byte lines of its Q and O rows, shared by neighbouring heads, are read
// and written once.
template <bool HEAD_MINOR = false>
__device__ __forceinline__ void decode_tile(const AttnMap& m, int heads, int L, int& h, int& s,
                                            int& j) {
  const int total = m.tile_start[m.n];
  int t;
  if (HEAD_MINOR) {
    t = L / heads;
    h = L - t * heads;
  } else {
    h = L / total;
    t = L - h * total;
  }
  s = 0;
#pragma unroll 1
  for (int i = 1; i < m.n; ++i) s += (t >= m.tile_start[i]) ? 1 : 0;
  j = t - m.tile_start[s];
}

// ROLE: 0 = self / joint attention, 1 = cross-attention to text (separate
// instances, so that profiles tell them apart).  QS: Q arrives already
// multiplied by scale_log2 (the model's projections write it so, rounding the
// scaled value once), else the scale is applied in fp32 to each score.
template <int HD, int NW, int ST, int ROLE, bool QS>
__global__ __launch_bounds__(NW * 64, 8 / NW) void attn_bf16_kernel(AttnMap map, int heads,
                                                           const bf16* __restrict__ Q, int ldq,
                                                           const bf16* __restrict__ K, int ldk,
                                                           const bf16* __restrict__ Vt, int ldvt,
                                                           bf16* __restrict__ O, int ldo,
                                                           float scale_log2) {
  constexpr int BQ = NW * 32, BKV = 64;
  // 16-wide chunks of the S^T = K Q^T contraction: d = 0 .. HD-1, then one
  // more slot (d = HD) that carries the softmax shift: K has 1 there and Q has
  // -m, so the MFMA itself returns s - m
  constexpr int DC = (HD + 1 + 15) / 16;
  constexpr int DT = (HD + 31) / 32;   // 32-row d tiles of O^T = V^T P^T
  constexpr int HDO = DT * 32;
  // row sums: a spare V^T row of ones where O^T has padding rows, else a
  // per-lane sum of the probabilities
  constexpr bool ONES = HD < HDO;
  constexpr int CPR = HD / 8;          // 16-byte chunks per K row
  constexpr int PK = 2 * HD;           // K row pitch in LDS (bytes)
  // K chunk slot swizzle for pitches that are multiples of 64 bytes: the 16
  // rows one fragment read touches then cover all 64 banks
  constexpr int KRS = (CPR == 4 || CPR == 8 || CPR == 16) ? 16 / CPR : 0;
  constexpr int KSTAGE = BKV * PK;     // bytes
  constexpr int VSTAGE = HDO * 128;    // V^T rows of 64 keys
  static_assert(HD % 8 == 0 && KSTAGE % 1024 == 0, "head dim");
  // the next tile's scores are computed one step ahead, so the ring needs a
  // stage for it besides the current tile's and the one being refilled
  static_assert(ST >= 3, "stages");
  __shared__ __attribute__((aligned(1024))) char smem[ST * (KSTAGE + VSTAGE)];

  // the wave index is uniform: keep it scalar so that per-wave choices below
  // are scalar branches
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int hh, s, j;
  decode_tile<ROLE == 1>(map, heads, xcd_remap_attn(blockIdx.x, gridDim.x), hh, s, j);
  const int q_beg = map.q_start[s], q_end = q_beg + map.q_len[s];
  // key tiles: those of segment 1, then those of segment 2
  const int k1 = map.k_start[s], n1 = map.k_len[s];
  const int k2 = map.k2_start[s], n2 = map.k2_len[s];
  const int t1 = (n1 + BKV - 1) / BKV, nt = t1 + (n2 + BKV - 1) / BKV;
  // tile ti starts at key (ti < t1 ? k1 : k2 - 64 t1) + 64 ti; only the last
  // tile of a segment can be ragged
  const int kb2 = k2 - t1 * BKV;
  const int rag1 = (n1 % BKV) ? t1 - 1 : -1, rag2 = (n2 % BKV) ? nt - 1 : -1;
  auto tile_kv0 = [&](int ti) { return (ti < t1 ? k1 : kb2) + ti * BKV; };
  auto tile_end = [&](int ti) { return ti < t1 ? k1 + n1 : k2 + n2; };
  auto tile_full = [&](int ti) { return ti != rag1 && ti != rag2; };
  // 32x32x16 MFMA lane roles: column (query) ql, k-half hl; C element 4i + jj
  // of a lane is row 8i + 4hl + jj
  const int ql = lane & 31, hl = lane >> 5;
  const int qr = q_beg + j * BQ + wave * 32 + ql;
  auto kst = [&](int st) { return smem + st * (KSTAGE + VSTAGE); };
  auto vst = [&](int st) { return smem + st * (KSTAGE + VSTAGE) + KSTAGE; };

  // Q fragments (B operand of S^T): query qr, d = 16c + 8hl .. +7, as stored.
  // Unless Q comes pre-scaled (QS), scores leave the MFMA in raw units and
  // the softmax scale log2(e)/sqrt(d) is applied in fp32 to each score before
  // its exponential: a scaled copy of a bf16 Q would be rounded a second time.
  // The shift slot d = HD is element 0 of chunk HD/16 in the lanes of half
  // (HD%16)/8
  constexpr int BC = HD / 16, BH = (HD % 16) / 8;
  bf16x8 qf[DC];
#pragma unroll
  for (int c = 0; c < DC; ++c) {
    const int d = c * 16 + hl * 8;
    qf[c] = bf16x8{};
    if (qr < q_end && d < HD) qf[c] = *(const bf16x8*)(Q + (size_t)qr * ldq + hh * HD + d);
  }
  auto init_ones = [&]() {
    // the ones row (V^T row HD) of every stage; the padding rows after it
    // only feed O^T rows that are never read
    if constexpr (ONES)
      for (int i = tid; i < ST * 64; i += NW * 64)
        ((bf16*)(vst(i >> 6) + HD * 128))[i & 63] = (bf16)1.f;
  };

  // Tile loads: HBM -> LDS directly (buffer_load_dwordx4 ... lds), instruction
  // c of a tensor's tile writes bytes 1024c .. +1023 of its part of the
  // stage, lane l 16 bytes at 16l.
  //   K: row r = key swap23(r), chunk slot swizzled; keys past the sequence
  //     are clamped to its last key (their scores are masked);
  //   V^T: row d, 128 bytes = 64 keys, chunk slot c ^ ((d>>1)&7); chunks
  //     wholly past the sequence are read from the tile's first chunk (their
  //     probabilities are 0).
  // Addresses: buffer resources based at K and V^T, the tile's position as
  // the scalar offset and per-lane 32-bit byte offsets.  The buffer form of
  // the LDS DMA, not the global one: the compiler counts an outstanding
  // global-form DMA as an out-of-order LDS event and then drains every LDS
  // fragment read with lgkmcnt(0), while the buffer form is tracked by vmcnt
  // alone, so the reads of the main loop get exact waits.  The launcher keeps
  // every offset below 2^31.
  // Only waves 0 .. NWD-1 issue loads -- the first half of them K, the second
  // half V^T, IPD instructions each -- so that the scalar work of a tile
  // (one M0 update per instruction) is not repeated by every wave: the CU's
  // scalar unit is shared by all its waves, which reach this point together.
  // Head dimensions of 128 and more keep 8 issuing waves (4 instructions
  // each), as the per-lane offsets of more instructions per wave would not
  // fit in the loop's registers.
  constexpr int NWD = NW < 4 ? NW : (CPR >= 16 ? NW : 4), WPT = NWD / 2;
  constexpr int IPD = (CPR + WPT - 1) / WPT;
  const bool dma_wave = wave < NWD, is_v = wave >= WPT;
  const int c_first = (wave % WPT) * IPD;
  const int n_w = dma_wave ? min(IPD, CPR - c_first) : 0;   // loads per tile
  auto k_lane = [&](int c, int& key, int& col) {   // K instruction c: key row, column
    const int o = c * 1024 + lane * 16;
    const int r = o / PK, slot = (o - r * PK) / 16;
    key = swap23(r);
    col = hh * HD + 8 * (KRS ? slot ^ ((r / KRS) & (CPR - 1)) : slot);
  };
  auto v_lane = [&](int c, int& row, int& key) {   // V^T instruction c: row, key
    const int o = c * 1024 + lane * 16, d = o / 128;
    row = hh * HD + d;
    key = 8 * ((lane & 7) ^ ((d >> 1) & 7));
  };
  uint32_t f_off[IPD];   // byte offset from the tile base (full tiles)
#pragma unroll
  for (int cc = 0; cc < IPD; ++cc) {
    const int c = min(c_first + cc, CPR - 1);
    int a, b;
    if (is_v) {
      v_lane(c, a, b);
      f_off[cc] = 2u * (uint32_t)(a * ldvt + b);
    } else {
      k_lane(c, a, b);
      f_off[cc] = 2u * (uint32_t)(a * ldk + b);
    }
  }
  // the launcher keeps every byte offset below 2^31, the extent given here
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      is_v ? (void*)Vt : (void*)K, 0, 0x7fffffff, kBufWord3);
  auto issue = [&](int ti) {
    if (!dma_wave) return;
    const int kv0 = tile_kv0(ti);
    const int soff = is_v ? 2 * kv0 : kv0 * (2 * ldk);   // the tile's byte offset
    char* lb = kst(ti % ST) + (is_v ? KSTAGE : 0) + c_first * 1024;
    auto load = [&](int cc, uint32_t off) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rsrc, (__attribute__((address_space(3))) void*)(lb + cc * 1024), 16, off, soff, 0, 0);
    };
    if (tile_full(ti)) {
#pragma unroll
      for (int cc = 0; cc < IPD; ++cc) {
        if (cc >= n_w) break;
        load(cc, f_off[cc]);
      }
      return;
    }
    // ragged tile: clamp keys past the sequence
    const int k_end = tile_end(ti);
#pragma unroll
    for (int cc = 0; cc < IPD; ++cc) {
      if (cc >= n_w) break;
      int a, b;
      if (is_v) {
        v_lane(c_first + cc, a, b);
        load(cc, 2u * (uint32_t)(a * ldvt + (kv0 + b < k_end ? b : 0)));
      } else {
        k_lane(c_first + cc, a, b);
        load(cc, 2u * (uint32_t)((min(kv0 + a, k_end - 1) - kv0) * ldk + b));
      }
    }
  };
  // K fragment (A operand) of key block kb, 16-wide d chunk c for this lane:
  // LDS row 32kb + ql, 16-byte chunk 2c + hl (zero past HD)
  bf16x8 kone = bf16x8{};      // the K side of the shift slot
  kone[0] = (bf16)1.f;
  // The chunk holding the shift slot (c = HD/16) takes the constant by a
  // per-lane select after an unmasked read: a lane-masked read would write
  // EXEC, which ends the compiler's scheduling region and keeps the
  // exponentials from interleaving with these MFMAs.
  auto kfrag = [&](int st, int kb, int c) {
    const int r = 32 * kb + ql;
    auto at = [&](int cc) {
      const int slot = KRS ? cc ^ ((r / KRS) & (CPR - 1)) : cc;
      return *(const bf16x8*)(kst(st) + r * PK + slot * 16);
    };
    if (c < BC) return at(2 * c + hl);
    if constexpr (CPR & 1) {
      // half 0: data chunk HD/8 - 1; half 1: the shift slot
      const bf16x8 v = at(2 * c);
      return hl ? kone : v;
    } else {
      // half 0: the shift slot; half 1: zero
      return hl ? bf16x8{} : kone;
    }
  };
  auto qk = [&](int ti, f32x16 (&sc)[2]) {
    const int st = ti % ST;
#pragma unroll
    for (int c = 0; c < DC; ++c) {
      bf16x8 kf[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) kf[kb] = kfrag(st, kb, c);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        sc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kb], qf[c],
                                                         c == 0 ? f32x16{} : sc[kb], 0, 0, 0);
    }
  };
  auto lane_max = [&](const f32x16 (&sc)[2]) {
    float m0 = fmaxf(sc[0][0], sc[0][1]), m1 = fmaxf(sc[1][0], sc[1][1]);
#pragma unroll
    for (int e = 2; e < 16; e += 2) {
      m0 = fmaxf(fmaxf(m0, sc[0][e]), sc[0][e + 1]);
      m1 = fmaxf(fmaxf(m1, sc[1][e]), sc[1][e + 1]);
    }
    return fmaxf(m0, m1);
  };

  // Online softmax with a lazily updated maximum m of the scores (kept
  // bf16-representable, as it rides in Q's shift slot): scores arrive as
  // S' = s - m and the probabilities are exp2(sc * S'), sc = 1 for a
  // pre-scaled Q, else scale_log2.  While no sc * S' exceeds 8 the stale
  // maximum is kept: probabilities stay <= 256 and the common scale cancels
  // between numerator and row sum.
  const float sc = QS ? 1.0f : scale_log2;
  const float lazy_thr = 8.0f / sc;   // 8 in log2 units
  f32x16 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) o[dt] = f32x16{};
  float m_ref = 0.f, l_run = 0.f;   // the m in Q's shift slot (0 before the first tile)

  // one tile: S^T of tile ti is in cur with lane maximum lm; the next tile's
  // S^T and lane maximum go to nxt / lm_nxt
  //
  // With ST >= 5 stages the workgroup synchronises once per two tiles (at
  // even ti): tiles ti+1 and ti+2 (read by the two steps' next-tile scores)
  // have landed, the ST-5 after them may still be in flight, and tiles
  // ti+ST-2 and ti+ST-1 go into the stages of ti-2 and ti-1, which every
  // wave has finished with.  With fewer stages it synchronises every tile:
  // tile ti+1 landed, ST-3 in flight, tile ti+ST-1 into the stage of ti-1.
  constexpr bool PAIR = ST >= 5;
  constexpr int YOUNG = PAIR ? ST - 5 : ST - 3;   // tiles left in flight
  static_assert((YOUNG + 2) * IPD < 64, "vmcnt");
  auto step = [&](int ti, f32x16 (&cur)[2], float& lm, f32x16 (&nxt)[2], float& lm_nxt,
                  bool sync) {
    if (!PAIR || sync) {
      // immediate counts in the steady state
      const int young = min(YOUNG, nt - (PAIR ? 3 : 2) - ti);
      if (!dma_wave) {
      } else if (young == YOUNG && n_w == IPD) {
        wait_vmcnt<YOUNG * IPD>();
      } else if (young == YOUNG && n_w == IPD - 1) {
        wait_vmcnt<YOUNG * (IPD - 1)>();
      } else {
        wait_vmcnt_dyn(young > 0 ? young * n_w : 0);
      }
      attn_barrier();
      if (PAIR && ti + ST - 2 < nt) issue(ti + ST - 2);
      if (ti + ST - 1 < nt) issue(ti + ST - 1);
    }
    // Up to head dimension 72: the slot schedule's constants, and its first
    // LA + 1 fragment reads (K of the next tile, d chunks 0 and 1), issued
    // before the maximum test below, which they do not depend on, so that
    // their LDS latency overlaps it
    constexpr bool SLOTS = DC <= 5;
    constexpr int NQK = 2 * DC, NPV = 4 * DT, NSL = NQK + NPV, LA = 3;
    constexpr int NE = NQK + 3 * DT;   // slots carrying exponentials
    const int stn = (ti + 1) % ST;
    const char* vb = vst(ti % ST);
    // slot sl's A operand: K of the next tile for sl < NQK, else V^T row
    // 32dt + ql, keys 16q + 8hl .. +7
    auto frag = [&](int sl) {
      if (sl < NQK) return kfrag(stn, sl & 1, sl >> 1);
      const int q = (sl - NQK) / DT, dt = (sl - NQK) % DT, row = dt * 32 + ql;
      return *(const bf16x8*)(vb + row * 128 + (((2 * q + hl) ^ ((row >> 1) & 7)) << 4));
    };
    bf16x8 fr[SLOTS ? NSL : 1];
    if constexpr (SLOTS) {
#pragma unroll
      for (int sl = 0; sl <= LA; ++sl) fr[sl] = frag(sl);
    }
    if (!tile_full(ti)) {
      const int kv0 = tile_kv0(ti), k_end = tile_end(ti);
      // ragged tile: mask the scores past the sequence.  V^T chunks wholly
      // past it were copied from the tile's first chunk, finite when the
      // sequence length is a multiple of 8.  Otherwise a chunk the sequence
      // ends inside holds bytes from beyond it (and may have been copied):
      // zero every column past the sequence (their probabilities are 0)
      if (k_end & 7) {
        const int c0 = k_end - kv0;
        char* vb = vst(ti % ST);
        for (int i = tid; i < HD * 64; i += NW * 64) {
          const int d = i >> 6, col = i & 63;
          if (col >= c0)
            *(bf16*)(vb + d * 128 + (((col >> 3) ^ ((d >> 1) & 7)) << 4) + (col & 7) * 2) =
                (bf16)0.f;
        }
        attn_barrier();
      }
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (kv0 + swap23(32 * kb + 8 * (e >> 2) + 4 * hl + (e & 3)) >= k_end)
            cur[kb][e] = -INFINITY;
      lm = lane_max(cur);
    }
    if (ti == 0 || __any(lm > lazy_thr)) {
      // new maximum: the query's 64 scores sit in lanes ql and ql + 32
      const float mx = fmaxf(lm, __shfl_xor(lm, 32, 64)) + m_ref;   // tile maximum
      const float m_old = ti == 0 ? -INFINITY : m_ref;
      const float m_new = (float)(bf16)fmaxf(m_old, mx);
      const float alpha = __builtin_amdgcn_exp2f(QS ? m_old - m_new : (m_old - m_new) * sc);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) cur[kb] -= (m_new - m_ref);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o[dt] *= alpha;
      l_run *= alpha;
      m_ref = m_new;
      if (hl == BH) qf[BC][0] = (bf16)(-m_new);
    }
    if constexpr (SLOTS) {
      // Straight-line part in a fixed issue order.  Slot s issues one MFMA --
      // the next tile's S^T for s < NQK (chunk s/2, key block s%2), else P V
      // for (key chunk, d tile) -- then its share of this tile's exponentials
      // and the LDS fragment read LA slots ahead.  A scheduling barrier between
      // slots keeps the exponentials spread over the MFMAs instead of bunched
      // (the compiler otherwise clusters them).  P chunk q is complete before
      // the first P V MFMA that uses it.  The slots from MX0 on, once the
      // next tile's S^T MFMAs have finished, also take the lane maximum of
      // those scores, a share per slot, off the path between tiles.  For the
      // last tile the "next" scores come from a stale stage and are never
      // used.
      constexpr int MX0 = NQK + 2, NMX = NSL - MX0;
      float pe[32];     // exponential i = P chunk i/8, element i%8
      bf16x8 pf[4];
      float psum = 0.f;
      float mx = -INFINITY;
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int sl = 0; sl < NSL; ++sl) {
        if (sl < NQK) {
          const int c = sl >> 1, kb = sl & 1;
          nxt[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[sl], qf[c],
                                                            c == 0 ? f32x16{} : nxt[kb], 0, 0, 0);
        } else {
          const int q = (sl - NQK) / DT, dt = (sl - NQK) % DT;
          o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[sl], pf[q], o[dt], 0, 0, 0);
        }
        const int e0 = sl < NE ? (32 * sl + NE - 1) / NE : 32;
        const int e1 = sl + 1 < NE ? (32 * (sl + 1) + NE - 1) / NE : 32;
#pragma unroll
        for (int i = e0; i < e1; ++i) {
          pe[i] = __builtin_amdgcn_exp2f(QS ? cur[i >> 4][i & 15] : cur[i >> 4][i & 15] * sc);
          if (!ONES) psum += pe[i];
          if ((i & 7) == 7)
#pragma unroll
            for (int e = 0; e < 8; ++e) pf[i >> 3][e] = (bf16)pe[(i & ~7) + e];
        }
        if (sl >= MX0) {
          const int v0 = 32 * (sl - MX0) / NMX, v1 = 32 * (sl - MX0 + 1) / NMX;
#pragma unroll
          for (int v = v0; v < v1; ++v) mx = fmaxf(mx, nxt[v >> 4][v & 15]);
          // keep the share in this slot (otherwise the chain is sunk to the
          // next tile's maximum test, in front of its first MFMA)
          asm volatile("" : "+v"(mx));
        }
        if (sl + LA + 1 < NSL) fr[sl + LA + 1] = frag(sl + LA + 1);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (!ONES) l_run += psum;
      lm_nxt = mx;
    } else {
      // larger head dimensions: the compiler's schedule (the fixed order
      // needs more registers than the loop has there) -- the next tile's
      // scores, then this tile's exponentials and P V
      qk(ti + 1, nxt);
      bf16x8 pf[4];
      float psum = 0.f;
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float x = cur[q >> 1][8 * (q & 1) + e];
          const float p = __builtin_amdgcn_exp2f(QS ? x : x * sc);
          if (!ONES) psum += p;
          pf[q][e] = (bf16)p;
        }
      if (!ONES) l_run += psum;
      const char* vb = vst(ti % ST);
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const int row = dt * 32 + ql;
          const bf16x8 vf =
              *(const bf16x8*)(vb + row * 128 + (((2 * q + hl) ^ ((row >> 1) & 7)) << 4));
          o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[q], o[dt], 0, 0, 0);
        }
      lm_nxt = lane_max(nxt);
    }
  };

  // prologue: the tiles before the first step's loads in flight, tile 0's
  // scores
  constexpr int PRE = PAIR ? ST - 2 : ST - 1;
#pragma unroll
  for (int ti = 0; ti < PRE; ++ti)
    if (ti < nt) issue(ti);
  init_ones();
  wait_vmcnt_dyn(n_w * (min(nt, PRE) - 1));
  attn_barrier();
  f32x16 sa[2], sb[2];
  float la, lb;
  qk(0, sa);
  la = lane_max(sa);
  for (int ti = 0; ti < nt; ti += 2) {
    step(ti, sa, la, sb, lb, true);
    if (ti + 1 < nt) step(ti + 1, sb, lb, sa, la, false);
  }

  float l;
  if (ONES) {
    // row HD of O^T = sum of the probabilities: tile HD/32, row r = HD%32 =
    // 8i + 4h + jj, held by the lanes of half h as element 4i + jj
    constexpr int R = HD % 32;
    l = __shfl(o[HD / 32][4 * (R / 8) + (R % 4)], ((R % 8) / 4) * 32 + ql, 64);
  } else {
    l = l_run + __shfl_xor(l_run, 32, 64);
  }
  if (qr >= q_end) return;
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
        *(bf16x4*)(O + (size_t)qr * ldo + hh * HD + d) = w;
      }
    }
}

// ---------------------------------------------------------------------------
// Cross-attention to a text of at most 128 keys (two key tiles).  Both tiles
// are loaded once into LDS, all scores are computed, and the softmax uses
// the exact row maximum (no running maximum, no rescaling, no next-tile
// lookahead).  A workgroup takes R consecutive query tiles of one head: the
// text's K / V^T stay in LDS from one to the next (reloaded only where the
// tiles cross into another sequence), and the next tile's Q fragments are
// fetched while this tile computes, so that its loads, its MFMAs and the
// previous tile's output stores overlap instead of the whole launch passing
// through them in step (with R = 1, one round of small workgroups does).
// The register and LDS footprint (40 KB at head dimension 72) lets four
// 4-wave workgroups share a CU at R = 1 and two at R > 1.  Workgroups of
// neighbouring heads take the same query tiles at the same time, so the
// 128-byte lines of the Q and O rows, shared by neighbouring heads, are read
// and written once.
// Layouts (K rows in swap23 key order, V^T chunk swizzle, ones row of V^T for
// the row sums) and the QS convention are those of attn_bf16_kernel.
template <int HD, int NW, bool QS, int R>
__global__ __launch_bounds__(NW * 64, (R > 1 ? 8 : (HD <= 72 ? 16 : 12)) / NW) void attn_cross_kernel(
    AttnMap map, int heads, const bf16* __restrict__ Q, int ldq, const bf16* __restrict__ K,
    int ldk, const bf16* __restrict__ Vt, int ldvt, bf16* __restrict__ O, int ldo,
    float scale_log2) {
  using X = XTile<HD>;
  constexpr int BQ = NW * 32, BKV = X::BKV, DC = X::DC, NI = X::NI;
  constexpr int KSTAGE = X::KSTAGE, VSTAGE = X::VSTAGE;
  // stage 0's V^T padding rows read stage 1's K rows, stage 1's this pad
  constexpr int VPAD = (X::HDO - X::VROWS) * 128;
  __shared__ __attribute__((aligned(1024))) char smem[2 * (KSTAGE + VSTAGE) + VPAD];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int total = map.tile_start[map.n];   // query tiles of all sequences
  const int L = xcd_remap_attn(blockIdx.x, gridDim.x);
  const int hh = L % heads, t_first = (L / heads) * R;
  const int ql = lane & 31, hl = lane >> 5;
  auto kst = [&](int t) { return smem + t * (KSTAGE + VSTAGE); };
  auto vst = [&](int t) { return smem + t * (KSTAGE + VSTAGE) + KSTAGE; };
  auto seq_of = [&](int t) {
    int s = 0;
#pragma unroll 1
    for (int i = 1; i < map.n; ++i) s += (t >= map.tile_start[i]) ? 1 : 0;
    return s;
  };

  // K / V^T tile loads of sequence s, the NI instructions of a tile spread
  // over the waves
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc((void*)K, 0, 0x7fffffff, kBufWord3);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc((void*)Vt, 0, 0x7fffffff, kBufWord3);
  auto load_kv = [&](int s) {
    const int k0 = map.k_start[s], k_end = k0 + map.k_len[s];
    const int nt = (map.k_len[s] + BKV - 1) / BKV;   // 1 or 2 (the launcher checks)
    for (int t = 0; t < nt; ++t) {
#pragma unroll
      for (int ii = 0; ii < (NI + NW - 1) / NW; ++ii) {
        const int i = wave + NW * ii;
        if (i >= NI) break;
        xattn_dma<HD>(rk, rv, i, k0 + t * BKV, k_end, hh, ldk, ldvt, kst(t), vst(t));
      }
    }
  };
  // after the loads of sequence s have landed
  auto fix_ragged = [&](int s) {
    const int nkeys = map.k_len[s];
    if (xattn_fix_ragged<HD>(vst((nkeys - 1) / BKV), nkeys, tid, NW * 64)) attn_barrier();
  };
  // Q fragments of query tile t (as stored): exactly DC loads per lane, from
  // a clamped row and column, so the vmcnt thresholds below can count them;
  // mask_q then zeroes the ones outside the tile, once the data are needed
  auto q_row = [&](int t, int& q_end) {
    const int s = seq_of(t);
    q_end = map.q_start[s] + map.q_len[s];
    return map.q_start[s] + (t - map.tile_start[s]) * BQ + wave * 32 + ql;
  };
  auto load_q = [&](int t, bf16x8 (&f)[DC]) {
    int q_end;
    const int qc = min(q_row(t, q_end), q_end - 1);
#pragma unroll
    for (int c = 0; c < DC; ++c)
      f[c] = *(const bf16x8*)(Q + (size_t)qc * ldq + hh * HD + min(c * 16 + hl * 8, HD - 8));
  };
  auto mask_q = [&](int t, const bf16x8 (&src)[DC], bf16x8 (&f)[DC]) {
    int q_end;
    const int qr = q_row(t, q_end);
#pragma unroll
    for (int c = 0; c < DC; ++c)
      f[c] = (qr < q_end && c * 16 + hl * 8 < HD) ? src[c] : bf16x8{};
  };

  int s_cur = seq_of(t_first);
  bf16x8 qf[DC], qn[DC];
  load_q(t_first, qn);
  load_kv(s_cur);
  const bool pre = R > 1 && t_first + 1 < total;
  bf16x8 qa[DC];
  if (pre) load_q(t_first + 1, qa);
  // the ones rows of both stages (the tile loads never write them)
  xattn_ones<HD>(vst(0), tid, NW * 64);
  xattn_ones<HD>(vst(1), tid, NW * 64);
  if (pre) wait_vmcnt<DC>();   // all but the next tile's Q
  else wait_vmcnt<0>();
  attn_barrier();
  fix_ragged(s_cur);
  mask_q(t_first, qn, qf);
#pragma unroll
  for (int c = 0; c < DC; ++c) qn[c] = qa[c];

  for (int r = 0; r < R; ++r) {
    const int tq = t_first + r;
    if (tq >= total) break;
    if (r > 0) {
      mask_q(tq, qn, qf);
      const int s_new = seq_of(tq);
      if (s_new != s_cur) {
        attn_barrier();   // every wave is done with the old K / V^T
        load_kv(s_new);
        wait_vmcnt<0>();
        attn_barrier();
        fix_ragged(s_new);
        s_cur = s_new;
      }
      if (r + 1 < R && tq + 1 < total) load_q(tq + 1, qn);
    }
    const int s = s_cur;
    const int q_end = map.q_start[s] + map.q_len[s];
    const int qr = map.q_start[s] + (tq - map.tile_start[s]) * BQ + wave * 32 + ql;
    bf16* const orow = O + (size_t)qr * ldo + hh * HD;
    xattn_wave<HD, QS>(kst(0), kst(1), vst(0), vst(1), map.k_len[s], qf, scale_log2, qr < q_end,
                       [&](int d, bf16x4 w) { *(bf16x4*)(orow + d) = w; });
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

// bf16: 8 waves x 32 queries per workgroup (stages: attn_stages).  Cross-attention to
// the text (two key tiles per query tile): 4 waves x 32 queries and 3 stages,
// so that two workgroups share a CU and one's loads overlap the other's
// compute.  Self / joint attention launches that would have fewer
// workgroups than CUs (short sequences, few heads) halve the workgroup, down
// to 2 waves.  fp32: 64 queries.
constexpr int kAttnWaves = 8;
// 8-wave workgroups: 5 stages (one barrier per two key tiles) up to head
// dimension 72; 4 above, where the loop's registers leave no room for the
// longer pipeline
template <int HD>
constexpr int attn_stages() {
  return HD <= 72 ? 5 : 4;
}
constexpr int kCrossWaves = 4, kCrossStages = 3;
void attention_tiles(AttnMap& m, bool bf16_io, int heads, int role) {
  auto fill = [&](int bq) {
    int t = 0;
    for (int s = 0; s < m.n; ++s) {
      m.tile_start[s] = t;
      t += (m.q_len[s] + bq - 1) / bq;
    }
    m.tile_start[m.n] = t;
    return (long)t * heads;
  };
  if (!bf16_io) {
    m.waves = 2;
    fill(64);
    return;
  }
  // default workgroup size; self / joint attention halves it while the
  // launch has fewer workgroups than CUs (256 on MI355X) -- cross-attention,
  // with two key tiles per query tile, measured slower with smaller groups
  int w = role == 1 ? kCrossWaves : kAttnWaves;
  long wgs = fill(32 * w);
  while (role == 0 && w > 2 && wgs < 256) {
    w /= 2;
    wgs = fill(32 * w);
  }
  m.waves = w;
}

template <int HD, bool QS>
static hipError_t launch_hd(bool bf16_io, int role, int heads, const AttnMap& map, const void* q,
                            int ldq, const void* k, int ldk, const void* v, int ldv, void* o,
                            int ldo, hipStream_t st) {
  const int tiles = map.tile_start[map.n] * heads;
  if (tiles == 0) return hipSuccess;
  if (bf16_io) {
    // tile loads address K and V^T with byte offsets below 2^31
    size_t k_rows = 0;
    for (int s = 0; s < map.n; ++s)
      k_rows = std::max(k_rows, (size_t)std::max(map.k_start[s] + map.k_len[s],
                                                 map.k2_start[s] + map.k2_len[s]));
    if ((size_t)2 * heads * HD * ldv > 0x7fffffff || (size_t)2 * (k_rows + 64) * ldk > 0x7fffffff)
      return hipErrorInvalidValue;
    const float scale_log2 = attn_q_scale(HD);
#define T2I_ATT(NW_, ST_, R_)                                                                   \
  hipLaunchKernelGGL((attn_bf16_kernel<HD, NW_, ST_, R_, QS>), dim3(tiles), dim3(NW_ * 64), 0, st, map, \
                     heads, (const bf16*)q, ldq, (const bf16*)k, ldk, (const bf16*)v, ldv,       \
                     (bf16*)o, ldo, scale_log2)
    // smaller workgroups (2 or 4 waves) share a CU and use a 3-stage ring
    if (role == 1) {
      // texts of at most 128 keys in one segment: the two-tile kernel
      bool short_text = map.waves == kCrossWaves;
      for (int s = 0; s < map.n && short_text; ++s)
        short_text = map.k_len[s] >= 1 && map.k_len[s] <= 128 && map.k2_len[s] == 0;
      // two query tiles per workgroup where the launch then still fills the
      // chip in one round at two workgroups per CU (1024 px with guidance:
      // 64 tiles x 16 heads -> 512 workgroups; measured 21.5 -> 20.2 us); a
      // second round of them (packed batches of ~1500 tile-head pairs)
      // measured slower than one tile per workgroup
      const int qt = map.tile_start[map.n];
      const long pairs = (long)((qt + 1) / 2) * heads;
      if (short_text && tiles >= 1024 && pairs <= 512) {
        hipLaunchKernelGGL((attn_cross_kernel<HD, kCrossWaves, QS, 2>),
                           dim3(((qt + 1) / 2) * heads), dim3(kCrossWaves * 64), 0, st, map, heads,
                           (const bf16*)q, ldq, (const bf16*)k, ldk, (const bf16*)v, ldv, (bf16*)o,
                           ldo, scale_log2);
      } else if (short_text) {
        hipLaunchKernelGGL((attn_cross_kernel<HD, kCrossWaves, QS, 1>), dim3(tiles),
                           dim3(kCrossWaves * 64), 0, st, map, heads, (const bf16*)q, ldq,
                           (const bf16*)k, ldk, (const bf16*)v, ldv, (bf16*)o, ldo, scale_log2);
      } else if (map.waves == kCrossWaves) T2I_ATT(kCrossWaves, kCrossStages, 1);
      else return hipErrorInvalidValue;
    } else {
      if (map.waves == kAttnWaves) T2I_ATT(kAttnWaves, attn_stages<HD>(), 0);
      else if (map.waves == 4) T2I_ATT(4, 3, 0);
      else if (map.waves == 2) T2I_ATT(2, 3, 0);
      else return hipErrorInvalidValue;
    }
#undef T2I_ATT
  } else {
    const float scale = 1.0f / sqrtf((float)HD);
    hipLaunchKernelGGL(attn_f32_kernel<HD>, dim3(tiles), dim3(64), 0, st, map, heads,
                       (const float*)q, ldq, (const float*)k, ldk, (const float*)v, ldv, (float*)o,
                       ldo, scale);
  }
  return hipGetLastError();
}

hipError_t launch_attention(bool bf16_io, int role, int heads, int head_dim, const AttnMap& map,
                            const void* q, int ldq, const void* k, int ldk, const void* v, int ldv,
                            void* o, int ldo, hipStream_t st, bool q_prescaled) {
#define T2I_HD(D_)                                                                             \
  case D_:                                                                                     \
    return q_prescaled && bf16_io                                                              \
               ? launch_hd<D_, true>(bf16_io, role, heads, map, q, ldq, k, ldk, v, ldv, o, ldo, st) \
               : launch_hd<D_, false>(bf16_io, role, heads, map, q, ldq, k, ldk, v, ldv, o, ldo, st);
  switch (head_dim) {
    T2I_HD(8)
    T2I_HD(32)
    T2I_HD(64)
    T2I_HD(72)
    T2I_HD(128)
    default: return hipErrorInvalidValue;
  }
#undef T2I_HD
}

}  // namespace t2i
