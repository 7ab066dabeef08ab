// HBM-bound kernels of the denoising step on gfx950: patch + position
// embedding, timestep sinusoid, LayerNorm fused with adaLN modulation, the
// final layer fused with unpatchify + classifier-free guidance + Euler update,
// and the step-skip cache reductions.
//
// Row kernels use one 64-lane wave per row with float4 loads (a row of
// D = 1152 floats is 4.5 KB: lane i reads float4 i, i+64, ...), so every load
// instruction of a wave covers 1 KB of contiguous memory.  Reductions run in
// registers with a fixed butterfly order, so results are bitwise reproducible.
#include <algorithm>

#include "t2i_internal.h"

namespace t2i {

constexpr int kMaxV4 = 12;   // float4 per lane: rows up to 3072 wide

// ---------------------------------------------------------------------------
// LayerNorm (biased variance, no affine) + modulation.

// Sum over the 64 lanes of a wave, the same value in every lane: DPP steps
// inside each 16-lane row, then the four row sums read out in a fixed order.
__device__ __forceinline__ float wave_sum_dpp(float v) {
  auto add_dpp = [](float x, int y) { return x + __int_as_float(y); };
  v = add_dpp(v, __builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));  // quad_perm 1,0,3,2
  v = add_dpp(v, __builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));  // quad_perm 2,3,0,1
  v = add_dpp(v, __builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x124, 0xF, 0xF, false)); // row_ror 4
  v = add_dpp(v, __builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xF, 0xF, false)); // row_ror 8
  const int b = __float_as_int(v);
  return (__int_as_float(__builtin_amdgcn_readlane(b, 0)) +
          __int_as_float(__builtin_amdgcn_readlane(b, 16))) +
         (__int_as_float(__builtin_amdgcn_readlane(b, 32)) +
          __int_as_float(__builtin_amdgcn_readlane(b, 48)));
}

// One wave per row, four rows per workgroup: many small independent waves
// keep enough loads in flight (the kernel is bound by memory latency).
constexpr int kLnRows = 4;

// NV: float4 per row known at compile time (0 = any width up to kMaxV4 * 256),
// so that registers are sized for the row.  The modulation rows are loaded
// together with the row, before the reductions that they do not depend on.
template <typename OutT, int NV>
__global__ __launch_bounds__(256) void ln_mod_kernel(const float* __restrict__ x, int ldx, int rows,
                                                     int D, const float* __restrict__ mod,
                                                     int ld_mod, int shift_off, int scale_off,
                                                     SeqMap map, OutT* __restrict__ out, int ldo,
                                                     float eps) {
  constexpr int NI = NV ? (NV + 63) / 64 : kMaxV4;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * kLnRows + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int nv = NV ? NV : D >> 2;
  const float4* xr = (const float4*)(x + (size_t)row * ldx);
  const float* md = mod + (size_t)map.modrow[seq_of_row(map, row)] * ld_mod;
  const float4* sh = (const float4*)(md + shift_off);
  const float4* sc = (const float4*)(md + scale_off);
  // (any-width instances load the modulation rows at their use, which keeps
  // their register count down)
  constexpr bool PRE = NV != 0;
  float4 v[NI], shv[PRE ? NI : 1], scv[PRE ? NI : 1];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int c = lane + 64 * i;
    if (c < nv) {
      v[i] = xr[c];
      if constexpr (PRE) {
        shv[i] = sh[c];
        scv[i] = sc[c];
      }
    }
  }
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int c = lane + 64 * i;
    if (c < nv) s += (v[i].x + v[i].y) + (v[i].z + v[i].w);
  }
  const float mean = wave_sum_dpp(s) / (float)D;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int c = lane + 64 * i;
    if (c < nv) {
      const float a = v[i].x - mean, b = v[i].y - mean, cc = v[i].z - mean, d = v[i].w - mean;
      q += (a * a + b * b) + (cc * cc + d * d);
    }
  }
  const float rstd = 1.0f / sqrtf(wave_sum_dpp(q) / (float)D + eps);
  OutT* orow = out + (size_t)row * ldo;
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int c = lane + 64 * i;
    if (c < nv) {
      const float4 a = PRE ? shv[PRE ? i : 0] : sh[c], b = PRE ? scv[PRE ? i : 0] : sc[c];
      const float y0 = (v[i].x - mean) * rstd * (1.f + b.x) + a.x;
      const float y1 = (v[i].y - mean) * rstd * (1.f + b.y) + a.y;
      const float y2 = (v[i].z - mean) * rstd * (1.f + b.z) + a.z;
      const float y3 = (v[i].w - mean) * rstd * (1.f + b.w) + a.w;
      if constexpr (sizeof(OutT) == 2)     // one 8-byte store of four bf16
        *(bf16x4*)(orow + 4 * c) = bf16x4{(bf16)y0, (bf16)y1, (bf16)y2, (bf16)y3};
      else
        *(float4*)(orow + 4 * c) = float4{y0, y1, y2, y3};
    }
  }
}

// RW consecutive rows per wave (D = 1152, RW = 2): the first row and the
// modulation rows are loaded first, then each row's successor before its
// reductions and stores, so the first row's arithmetic starts as early as
// possible and reads and writes overlap.  With two rows per wave the launch
// fits one round of the chip's wave slots (one wave per row leaves a partial
// second round; more rows per wave measured slower: 4 rows as fast as the
// two-row kernel that loaded both rows first, 8 rows 25 % slower).  The
// modulation rows are reloaded only when the sequence changes.  Per-row
// arithmetic as in ln_mod_kernel (bitwise equal).
template <typename OutT, int NV, int RW>
__global__ __launch_bounds__(256) void ln_modr_kernel(const float* __restrict__ x, int ldx, int rows,
                                                      int D, const float* __restrict__ mod,
                                                      int ld_mod, int shift_off, int scale_off,
                                                      SeqMap map, OutT* __restrict__ out, int ldo,
                                                      float eps) {
  constexpr int NI = (NV + 63) / 64;
  const int lane = threadIdx.x & 63;
  const int r0 = (blockIdx.x * kLnRows + (threadIdx.x >> 6)) * RW;
  if (r0 >= rows) return;
  const int rn = min(RW, rows - r0);
  float4 v[2][NI], shv[NI], scv[NI];
  auto load_row = [&](float4 (&b)[NI], int row) {
    const float4* xr = (const float4*)(x + (size_t)row * ldx);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int c = lane + 64 * i;
      if (c < NV) b[i] = xr[c];
    }
  };
  auto load_mod = [&](int mr) {
    const float4* sh = (const float4*)(mod + (size_t)mr * ld_mod + shift_off);
    const float4* sc = (const float4*)(mod + (size_t)mr * ld_mod + scale_off);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int c = lane + 64 * i;
      if (c < NV) {
        shv[i] = sh[c];
        scv[i] = sc[c];
      }
    }
  };
  load_row(v[0], r0);
  int mcur = map.modrow[seq_of_row(map, r0)];
  load_mod(mcur);
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    if (r >= rn) break;
    if (r + 1 < rn) load_row(v[(r + 1) & 1], r0 + r + 1);
    if (r > 0) {
      const int mr = map.modrow[seq_of_row(map, r0 + r)];
      if (mr != mcur) {
        load_mod(mr);
        mcur = mr;
      }
    }
    const float4* vr = v[r & 1];
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int c = lane + 64 * i;
      if (c < NV) s += (vr[i].x + vr[i].y) + (vr[i].z + vr[i].w);
    }
    const float mean = wave_sum_dpp(s) / (float)D;
    float q = 0.f;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int c = lane + 64 * i;
      if (c < NV) {
        const float a = vr[i].x - mean, b = vr[i].y - mean, cc = vr[i].z - mean, d = vr[i].w - mean;
        q += (a * a + b * b) + (cc * cc + d * d);
      }
    }
    const float rstd = 1.0f / sqrtf(wave_sum_dpp(q) / (float)D + eps);
    OutT* orow = out + (size_t)(r0 + r) * ldo;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int c = lane + 64 * i;
      if (c < NV) {
        const float4 a = shv[i], b = scv[i];
        const float y0 = (vr[i].x - mean) * rstd * (1.f + b.x) + a.x;
        const float y1 = (vr[i].y - mean) * rstd * (1.f + b.y) + a.y;
        const float y2 = (vr[i].z - mean) * rstd * (1.f + b.z) + a.z;
        const float y3 = (vr[i].w - mean) * rstd * (1.f + b.w) + a.w;
        if constexpr (sizeof(OutT) == 2)
          *(bf16x4*)(orow + 4 * c) = bf16x4{(bf16)y0, (bf16)y1, (bf16)y2, (bf16)y3};
        else
          *(float4*)(orow + 4 * c) = float4{y0, y1, y2, y3};
      }
    }
  }
}

hipError_t launch_ln_modulate(bool bf16_out, int rows, int D, const float* x, int ldx,
                              const float* mod, int ld_mod, int shift_off, int scale_off,
                              const SeqMap& map, void* out, int ldo, float eps, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  dim3 grid((rows + kLnRows - 1) / kLnRows), block(256);
#define T2I_LN(T_, NV_)                                                                      \
  hipLaunchKernelGGL((ln_mod_kernel<T_, NV_>), grid, block, 0, st, x, ldx, rows, D, mod, ld_mod, \
                     shift_off, scale_off, map, (T_*)out, ldo, eps)
  if (bf16_out) {
    if (D == 1152) {
      constexpr int RW = 2;
      hipLaunchKernelGGL((ln_modr_kernel<bf16, 288, RW>), dim3((rows + RW * kLnRows - 1) / (RW * kLnRows)),
                         block, 0, st, x, ldx, rows, D, mod, ld_mod, shift_off, scale_off, map,
                         (bf16*)out, ldo, eps);
      return hipGetLastError();
    }
    if (D == 3072) T2I_LN(bf16, 768);
    else T2I_LN(bf16, 0);
  } else {
    T2I_LN(float, 0);
  }
#undef T2I_LN
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Patchify + patch embedding (+ 2D sin-cos position embedding).
// Token i*(w/p)+j of a request reads latent [c, i*p+a, j*p+b] as feature
// (a*p+b)*C+c.  Writes x0 (one copy) and `copies` copies into x (one per
// guidance branch, branch-major).
//
// pe_table_kernel: tab[pos * qd + f] = (sin, cos)(pos * 10000^(-f/qd)) in fp64,
// qd = D/4.  embed_kernel: a workgroup takes kEmbTok tokens x 256 channels;
// the tokens' patches are staged in LDS, each thread keeps its channel's
// weight row in registers.  The first D/2 channels add the row's sin-cos
// embedding, the last D/2 the column's; within a half the first D/4 are sin,
// the next D/4 cos.

__global__ void pe_table_kernel(float2* __restrict__ tab, int npos, int qd) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= npos * qd) return;
  const int pos = i / qd, f = i - pos * qd;
  const double ang = (double)pos * pow(10000.0, -(double)f / (double)qd);
  tab[i] = float2{(float)sin(ang), (float)cos(ang)};
}

// 8 tokens per workgroup: 2560 workgroups for 4096 tokens (measured against
// 32: 29.5 -> 24.8 us at 4096 tokens x 2 branches, 23.7 -> 13.7 us at 1024
// tokens), the stores spread evenly over the CUs
constexpr int kEmbTok = 8;

// PT: patch features p*p*C known at compile time (16, 64), else 0 (any
// P <= 64): with constant trip counts the weights load as 16-byte vectors and
// the patch rows as float4, with no per-feature branches.
template <typename TW, int PT>
__global__ __launch_bounds__(256) void embed_kernel(const float* __restrict__ lat, ReqMap rm,
                                                    const TW* __restrict__ w_pe,
                                                    const TW* __restrict__ b_pe, int D, int C,
                                                    int p, const float2* __restrict__ pe,
                                                    float* __restrict__ x0, float* __restrict__ x,
                                                    int copies) {
  // rows padded to 68 floats: 16-byte aligned, and neighbouring rows start
  // four banks apart
  __shared__ __attribute__((aligned(16))) float patch[kEmbTok][68];
  __shared__ int grid_pos[kEmbTok][2];
  __shared__ long long tok_base[kEmbTok];
  __shared__ int tok_w[kEmbTok], tok_hw[kEmbTok];
  const int P = PT ? PT : p * p * C;
  const int T = rm.tokens_total;
  const int t0 = blockIdx.x * kEmbTok, d = blockIdx.y * 256 + threadIdx.x;
  // each token's patch origin in its request's latent, once
  if (threadIdx.x < kEmbTok) {
    const int t = threadIdx.x, tok = t0 + t;
    long long base = -1;
    int W = 0, HW = 0;
    if (tok < T) {
      const int r = req_of_token(rm, tok);
      const int lt = tok - rm.tok_off[r];
      W = rm.w[r];
      HW = rm.h[r] * W;
      const int gw = W / p, gi = lt / gw, gj = lt - gi * gw;
      base = rm.lat_off[r] + (long long)(gi * p) * W + gj * p;
      grid_pos[t][0] = gi;
      grid_pos[t][1] = gj;
    }
    tok_base[t] = base;
    tok_w[t] = W;
    tok_hw[t] = HW;
  }
  __syncthreads();
  // gather element (t, k = (a p + b) C + c) in the order (c, a, t, b): the
  // pixels of neighbouring threads are neighbours in a latent row
  for (int i = threadIdx.x; i < kEmbTok * P; i += 256) {
    const int b = i % p, rest = i / p;
    const int t = rest % kEmbTok, ca = rest / kEmbTok;
    const int a = ca % p, c = ca / p;
    float v = 0.f;
    if (tok_base[t] >= 0)
      v = lat[tok_base[t] + (long long)c * tok_hw[t] + (long long)a * tok_w[t] + b];
    patch[t][(a * p + b) * C + c] = v;
  }
  __syncthreads();
  if (d >= D) return;
  constexpr int NW = PT ? PT : 64;
  float w[NW];
  if constexpr (PT > 0 && sizeof(TW) == 2) {
#pragma unroll
    for (int k8 = 0; k8 < PT / 8; ++k8) {
      const bf16x8 q = *(const bf16x8*)(w_pe + (size_t)d * PT + 8 * k8);
#pragma unroll
      for (int e = 0; e < 8; ++e) w[8 * k8 + e] = (float)q[e];
    }
  } else {
#pragma unroll
    for (int k = 0; k < NW; ++k) w[k] = k < P ? to_f32(w_pe[(size_t)d * P + k]) : 0.f;
  }
  const float bias = to_f32(b_pe[d]);
  const int half = D / 2, qd = D / 4, kk = d % half, f = kk % qd;
  for (int t = 0; t < kEmbTok; ++t) {
    const int tok = t0 + t;
    if (tok >= T) break;
    float acc = bias;
    if constexpr (PT > 0) {
#pragma unroll
      for (int k4 = 0; k4 < PT / 4; ++k4) {
        const float4 pv = *(const float4*)&patch[t][4 * k4];
        acc = fmaf(w[4 * k4 + 0], pv.x, acc);
        acc = fmaf(w[4 * k4 + 1], pv.y, acc);
        acc = fmaf(w[4 * k4 + 2], pv.z, acc);
        acc = fmaf(w[4 * k4 + 3], pv.w, acc);
      }
    } else {
#pragma unroll
      for (int k = 0; k < 64; ++k)
        if (k < P) acc = fmaf(w[k], patch[t][k], acc);
    }
    if (pe) {
      const float2 sc = pe[grid_pos[t][d < half ? 0 : 1] * qd + f];
      acc += kk < qd ? sc.x : sc.y;
    }
    x0[(size_t)tok * D + d] = acc;
    for (int cp = 0; cp < copies; ++cp) x[((size_t)cp * T + tok) * D + d] = acc;
  }
}

hipError_t launch_embed(const float* lat, const ReqMap& rm, const void* w_pe, const void* b_pe,
                        bool w_bf16, int D, int C, int p, float2* pe_table, int pe_npos,
                        float* x0, float* x, int copies, hipStream_t st) {
  if (rm.tokens_total == 0) return hipSuccess;
  if (pe_table) {
    const int n = pe_npos * (D / 4);
    hipLaunchKernelGGL(pe_table_kernel, dim3((n + 255) / 256), dim3(256), 0, st, pe_table, pe_npos,
                       D / 4);
  }
  dim3 grid((rm.tokens_total + kEmbTok - 1) / kEmbTok, (D + 255) / 256);
  const int P = p * p * C;
#define T2I_EMB(TW_, PT_)                                                                     \
  hipLaunchKernelGGL((embed_kernel<TW_, PT_>), grid, dim3(256), 0, st, lat, rm, (const TW_*)w_pe, \
                     (const TW_*)b_pe, D, C, p, pe_table, x0, x, copies)
  if (w_bf16) {
    if (P == 16) T2I_EMB(bf16, 16);
    else if (P == 64) T2I_EMB(bf16, 64);
    else T2I_EMB(bf16, 0);
  } else {
    if (P == 16) T2I_EMB(float, 16);
    else T2I_EMB(float, 0);
  }
#undef T2I_EMB
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Timestep sinusoid: row r, s = t_scale * t[r]: [cos(s f_k) | sin(s f_k)],
// f_k = exp(-ln(10000) k / half), evaluated in fp64.

__global__ void timestep_freq_kernel(TVals tv, int freq_dim, double t_scale,
                                     float* __restrict__ out) {
  const int half = freq_dim / 2;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= tv.n * freq_dim) return;
  const int r = idx / freq_dim, k = idx - r * freq_dim;
  const int kk = k < half ? k : k - half;
  const double f = exp(-log(10000.0) * (double)kk / (double)half);
  const double a = t_scale * tv.t[r] * f;
  out[idx] = (float)(k < half ? cos(a) : sin(a));
}

hipError_t launch_timestep_freq(const double* t, int rows, int freq_dim, double t_scale,
                                float* out, hipStream_t st) {
  for (int r0 = 0; r0 < rows; r0 += kTValsChunk) {
    TVals tv;
    tv.n = std::min(kTValsChunk, rows - r0);
    for (int i = 0; i < tv.n; ++i) tv.t[i] = t[r0 + i];
    const int n = tv.n * freq_dim;
    hipLaunchKernelGGL(timestep_freq_kernel, dim3((n + 255) / 256), dim3(256), 0, st, tv, freq_dim,
                       t_scale, out + (size_t)r0 * freq_dim);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// dst[r][:] = src[:] (bf16 or fp32 rows of width D)
__global__ void broadcast_rows_kernel(const uint16_t* __restrict__ src16,
                                      const float* __restrict__ src32, int rows, int D,
                                      uint16_t* __restrict__ dst16, float* __restrict__ dst32) {
  const long n = (long)rows * D;
  for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
    const int d = (int)(i % D);
    if (src16) dst16[i] = src16[d];
    else dst32[i] = src32[d];
  }
}

hipError_t launch_broadcast_rows(const void* src, bool bf16_io, int rows, int D, void* dst,
                                 hipStream_t st) {
  const long n = (long)rows * D;
  if (n == 0) return hipSuccess;
  const int grid = (int)std::min<long>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(broadcast_rows_kernel, dim3(grid), dim3(256), 0, st,
                     bf16_io ? (const uint16_t*)src : nullptr, bf16_io ? nullptr : (const float*)src,
                     rows, D, bf16_io ? (uint16_t*)dst : nullptr, bf16_io ? nullptr : (float*)dst);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// 2D rotary position embedding of the image tokens (joint-attention model).

__global__ void rope_table_kernel(float2* __restrict__ tab, int npos, int q) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= npos * q) return;
  const int pos = i / q, j = i - pos * q;
  const double ang = (double)pos * pow(10000.0, -(double)j / (double)q);
  tab[i] = float2{(float)cos(ang), (float)sin(ang)};
}

hipError_t launch_rope_table(float2* table, int npos, int q, hipStream_t st) {
  const int n = npos * q;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(rope_table_kernel, dim3((n + 255) / 256), dim3(256), 0, st, table, npos, q);
  return hipGetLastError();
}

// one thread per (row, head, half, pair): rotates the q pair and the k pair
__global__ void rope_apply_kernel(bf16* __restrict__ qk, int ld, int row0, ReqMap rm, int heads,
                                  int hd, int patch, const float2* __restrict__ tab) {
  const int q = hd / 4;
  const long per_row = (long)heads * 2 * q;
  const long total = (long)rm.tokens_total * rm.branches * per_row;
  const int D = heads * hd;
  for (long i = blockIdx.x * 256L + threadIdx.x; i < total; i += (long)gridDim.x * 256) {
    const long row = i / per_row;
    int rem = (int)(i - row * per_row);
    const int h = rem / (2 * q);
    rem -= h * 2 * q;
    const int half = rem / q, j = rem - half * q;
    const int tok = (int)(row % rm.tokens_total);
    const int r = req_of_token(rm, tok);
    const int lt = tok - rm.tok_off[r];
    const int gw = rm.w[r] / patch;
    const int pos = half ? lt % gw : lt / gw;
    const float2 cs = tab[pos * q + j];
    bf16* base = qk + (size_t)(row0 + row) * ld + h * hd + half * (hd / 2) + 2 * j;
#pragma unroll
    for (int part = 0; part < 2; ++part) {   // q, then k (D columns further)
      bf16* pp = base + part * D;
      const float a = (float)pp[0], b = (float)pp[1];
      pp[0] = (bf16)(a * cs.x - b * cs.y);
      pp[1] = (bf16)(a * cs.y + b * cs.x);
    }
  }
}

// Head dims that are multiples of 16: one thread per (row, head, half, group
// of 4 pairs) moves 16 bytes of q and of k at a time, with 32-bit index math;
// each pair is rotated exactly as in rope_apply_kernel.
__global__ void rope_apply4_kernel(bf16* __restrict__ qk, int ld, int row0, ReqMap rm, int heads,
                                   int hd, int patch, const float2* __restrict__ tab) {
  const int q = hd / 4, g = q / 4;
  const int per_row = heads * 2 * g;
  const int T = rm.tokens_total;
  const int total = T * rm.branches * per_row;
  const int D = heads * hd;
  for (int i = blockIdx.x * 256 + threadIdx.x; i < total; i += gridDim.x * 256) {
    const int row = i / per_row;
    int rem = i - row * per_row;
    const int h = rem / (2 * g);
    rem -= h * 2 * g;
    const int half = rem / g, jg = rem - half * g;
    const int tok = row >= T ? row - T : row;   // branch-major rows, two branches at most
    const int r = req_of_token(rm, tok);
    const int lt = tok - rm.tok_off[r];
    const int gw = rm.w[r] / patch;
    const int pos = half ? lt % gw : lt / gw;
    const float2* cs = tab + pos * q + 4 * jg;
    bf16* base = qk + (size_t)(row0 + row) * ld + h * hd + half * (hd / 2) + 8 * jg;
#pragma unroll
    for (int part = 0; part < 2; ++part) {   // q, then k (D columns further)
      bf16x8* pp = (bf16x8*)(base + part * D);
      const bf16x8 v = *pp;
      bf16x8 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float2 c = cs[e];
        const float a = (float)v[2 * e], b = (float)v[2 * e + 1];
        o[2 * e] = (bf16)(a * c.x - b * c.y);
        o[2 * e + 1] = (bf16)(a * c.y + b * c.x);
      }
      *pp = o;
    }
  }
}

hipError_t launch_rope_apply(bf16* qk, int ld, int row0, const ReqMap& rm, int heads, int head_dim,
                             int patch, const float2* table, hipStream_t st) {
  const long total = (long)rm.tokens_total * rm.branches * heads * (head_dim / 2);
  if (total == 0) return hipSuccess;
  if (head_dim % 16 == 0 && rm.branches <= 2 && ld % 8 == 0 && ((uintptr_t)qk % 16) == 0 &&
      total / 4 < (1L << 30)) {
    const int grid = (int)std::min<long>((total / 4 + 255) / 256, 16384);
    hipLaunchKernelGGL(rope_apply4_kernel, dim3(grid), dim3(256), 0, st, qk, ld, row0, rm, heads,
                       head_dim, patch, table);
    return hipGetLastError();
  }
  const int grid = (int)std::min<long>((total + 255) / 256, 16384);
  hipLaunchKernelGGL(rope_apply_kernel, dim3(grid), dim3(256), 0, st, qk, ld, row0, rm, heads,
                     head_dim, patch, table);
  return hipGetLastError();
}

// LoRA merge: a thread owns one input column i and keeps A[:, i] in
// registers; the workgroup walks kLoraRows output rows, B's rows staged in LDS.
// RK (16 / 32 / 64 / 128) is the rank rounded up; the padding is zero.
constexpr int kLoraRows = 64, kLoraMaxRank = 128;

template <typename T, int RK>
__global__ __launch_bounds__(256) void lora_merge_kernel(int n_out, int n_in, int rank, float alpha,
                                                         T* __restrict__ W, int ldw,
                                                         const T* __restrict__ A,
                                                         const T* __restrict__ B) {
  __shared__ float brow[kLoraRows][RK];
  const int i = blockIdx.x * 256 + threadIdx.x;
  const int o0 = blockIdx.y * kLoraRows;
  for (int e = threadIdx.x; e < kLoraRows * RK; e += 256) {
    const int r = e / RK, k = e - r * RK;
    brow[r][k] = (o0 + r < n_out && k < rank) ? to_f32(B[(size_t)(o0 + r) * rank + k]) : 0.f;
  }
  __syncthreads();
  if (i >= n_in) return;
  float a[RK];
#pragma unroll
  for (int k = 0; k < RK; ++k) a[k] = k < rank ? to_f32(A[(size_t)k * n_in + i]) : 0.f;
  const int rows = min(kLoraRows, n_out - o0);
  // 16 rows at a time: their W elements are loaded together (independent
  // loads in flight), updated, stored
  for (int r0 = 0; r0 < rows; r0 += 16) {
    float wv[16];
#pragma unroll
    for (int j = 0; j < 16; ++j)
      wv[j] = r0 + j < rows ? to_f32(W[(size_t)(o0 + r0 + j) * ldw + i]) : 0.f;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      float acc = 0.f;
#pragma unroll
      for (int k = 0; k < RK; ++k) acc = fmaf(brow[r0 + j][k], a[k], acc);
      if (r0 + j < rows) W[(size_t)(o0 + r0 + j) * ldw + i] = from_f32<T>(fmaf(alpha, acc, wv[j]));
    }
  }
}

// bf16 LoRA merge on MFMA.  A workgroup (4 waves) owns a 64-row x 128-column
// tile of W.  It first issues the loads of its W tile (16 bytes per lane,
// rows contiguous, four per thread, so the HBM reads are in flight from the
// start), then stages the tile's rank slice of B [64][RK] and of A,
// transposed to [128][RK] (k contiguous, as both MFMA operands want it), in
// LDS, zero-padded past `rank`; each wave computes two 32x32 tiles of B A on
// v_mfma_f32_32x32x16_bf16 (fp32 accumulation over the rank), writes them to
// LDS as fp32, and every thread then finishes its W chunks: W + alpha (B A),
// rounded once to bf16.  Needs n_in % 8 == 0, ldw % 8 == 0 and 16-byte
// aligned W and A rows (the launcher checks and falls back otherwise).
constexpr int kLoraTM = 64, kLoraTN = 128;

template <int RK>
__global__ __launch_bounds__(256) void lora_merge_mfma_kernel(int n_out, int n_in, int rank,
                                                              float alpha, LoraGroup g, int ldw) {
  // weight blockIdx.z of the group
  bf16* __restrict__ W = (bf16*)g.W[blockIdx.z];
  const bf16* __restrict__ A = (const bf16*)g.A[blockIdx.z];
  const bf16* __restrict__ B = (const bf16*)g.B[blockIdx.z];
  constexpr int KP = RK + 8;                         // LDS row pitch of the operands (bf16)
  constexpr int PP = kLoraTN + 4;                    // LDS row pitch of the product (fp32)
  constexpr int OPS = (kLoraTM + kLoraTN) * KP * 2;  // operand bytes
  constexpr int PRB = kLoraTM * PP * 4;              // product bytes
  __shared__ __attribute__((aligned(16))) char smem[OPS > PRB ? OPS : PRB];
  bf16* Bs = (bf16*)smem;                  // [64][KP]
  bf16* At = Bs + kLoraTM * KP;            // [128][KP]
  float* Ps = (float*)smem;                // [64][PP], after the MFMAs
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int o0 = blockIdx.y * kLoraTM, i0 = blockIdx.x * kLoraTN;

  // this thread's W chunks: row (tid >> 4) + 16 c, 8 columns at 8 (tid & 15)
  constexpr int NC = kLoraTM * kLoraTN / 8 / 256;
  const int cc = (tid & 15) * 8;
  bf16x8 wv[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int o = o0 + (tid >> 4) + 16 * c, i = i0 + cc;
    wv[c] = bf16x8{};
    if (o < n_out && i < n_in) wv[c] = *(const bf16x8*)(W + (size_t)o * ldw + i);
  }
  // operands into LDS, zero past rank / the matrix edges
  for (int e = tid; e < kLoraTM * (RK / 8); e += 256) {
    const int r = e / (RK / 8), k = (e - r * (RK / 8)) * 8;
    bf16x8 v = bf16x8{};
    if (o0 + r < n_out)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (k + j < rank) v[j] = B[(size_t)(o0 + r) * rank + k + j];
    *(bf16x8*)(Bs + r * KP + k) = v;
  }
  for (int e = tid; e < RK * (kLoraTN / 8); e += 256) {
    const int k = e / (kLoraTN / 8), c = (e - k * (kLoraTN / 8)) * 8;
    bf16x8 v = bf16x8{};
    if (k < rank && i0 + c < n_in) v = *(const bf16x8*)(A + (size_t)k * n_in + i0 + c);
#pragma unroll
    for (int j = 0; j < 8; ++j) At[(c + j) * KP + k] = v[j];
  }
  __syncthreads();
  // wave w: rows 32 (w & 1) .., columns 64 (w >> 1) .. (two 32-wide tiles)
  const int l32 = lane & 31, hl = lane >> 5;
  const int ro = 32 * (wave & 1), co = 64 * (wave >> 1);
  f32x16 acc[2] = {f32x16{}, f32x16{}};
#pragma unroll
  for (int k = 0; k < RK; k += 16) {
    const bf16x8 bo = *(const bf16x8*)(Bs + (ro + l32) * KP + k + 8 * hl);
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const bf16x8 ai = *(const bf16x8*)(At + (co + 32 * t + l32) * KP + k + 8 * hl);
      acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bo, ai, acc[t], 0, 0, 0);
    }
  }
  __syncthreads();   // the operands are no longer read: the product takes their place
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e)
      Ps[(ro + 8 * (e >> 2) + 4 * hl + (e & 3)) * PP + co + 32 * t + l32] = acc[t][e];
  __syncthreads();
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int r = (tid >> 4) + 16 * c, o = o0 + r, i = i0 + cc;
    if (o >= n_out || i >= n_in) continue;
    const float4 p0 = *(const float4*)(Ps + r * PP + cc);
    const float4 p1 = *(const float4*)(Ps + r * PP + cc + 4);
    const float pv[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
    bf16x8 out;
#pragma unroll
    for (int j = 0; j < 8; ++j) out[j] = (bf16)fmaf(alpha, pv[j], (float)wv[c][j]);
    *(bf16x8*)(W + (size_t)o * ldw + i) = out;
  }
}

template <typename T>
static hipError_t lora_dispatch(int n_out, int n_in, int rank, float alpha, void* W, int ldw,
                                const void* A, const void* B, hipStream_t st) {
  dim3 grid((n_in + 255) / 256, (n_out + kLoraRows - 1) / kLoraRows);
#define T2I_LORA(RK_)                                                                        \
  hipLaunchKernelGGL((lora_merge_kernel<T, RK_>), grid, dim3(256), 0, st, n_out, n_in, rank, \
                     alpha, (T*)W, ldw, (const T*)A, (const T*)B)
  if (rank <= 16) T2I_LORA(16);
  else if (rank <= 32) T2I_LORA(32);
  else if (rank <= 64) T2I_LORA(64);
  else T2I_LORA(128);
#undef T2I_LORA
  return hipGetLastError();
}

hipError_t launch_lora_merge(bool bf16_io, int n_out, int n_in, int rank, float alpha, void* W,
                             int ldw, const void* A, const void* B, hipStream_t st) {
  if (n_out <= 0 || n_in <= 0) return hipSuccess;
  if (rank < 1 || rank > kLoraMaxRank) return hipErrorInvalidValue;
  LoraGroup g;
  g.W[0] = W;
  g.A[0] = A;
  g.B[0] = B;
  return launch_lora_merge_group(bf16_io, 1, n_out, n_in, rank, alpha, g, ldw, st);
}

hipError_t launch_lora_merge_group(bool bf16_io, int n, int n_out, int n_in, int rank,
                                   float alpha, const LoraGroup& g, int ldw, hipStream_t st) {
  if (n <= 0 || n_out <= 0 || n_in <= 0) return hipSuccess;
  if (n > kMaxGroups || rank < 1 || rank > kLoraMaxRank) return hipErrorInvalidValue;
  bool vec = bf16_io && n_in % 8 == 0 && ldw % 8 == 0;
  for (int i = 0; i < n; ++i)
    vec = vec && (uintptr_t)g.W[i] % 16 == 0 && (uintptr_t)g.A[i] % 16 == 0;
  if (vec) {
    dim3 grid((n_in + kLoraTN - 1) / kLoraTN, (n_out + kLoraTM - 1) / kLoraTM, n);
#define T2I_LORA_MF(RK_)                                                                       \
  hipLaunchKernelGGL((lora_merge_mfma_kernel<RK_>), grid, dim3(256), 0, st, n_out, n_in, rank, \
                     alpha, g, ldw)
    if (rank <= 16) T2I_LORA_MF(16);
    else if (rank <= 32) T2I_LORA_MF(32);
    else if (rank <= 64) T2I_LORA_MF(64);
    else T2I_LORA_MF(128);
#undef T2I_LORA_MF
    return hipGetLastError();
  }
  for (int i = 0; i < n; ++i) {
    hipError_t e = bf16_io ? lora_dispatch<bf16>(n_out, n_in, rank, alpha, g.W[i], ldw, g.A[i],
                                                 g.B[i], st)
                           : lora_dispatch<float>(n_out, n_in, rank, alpha, g.W[i], ldw, g.A[i],
                                                  g.B[i], st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

__global__ void add_inplace_kernel(float* __restrict__ x, const float* __restrict__ r, size_t n) {
  for (size_t i = blockIdx.x * 256ul + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) x[i] += r[i];
}

hipError_t launch_add_inplace(float* x, const float* r, size_t n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  const int grid = (int)std::min<size_t>((n + 255) / 256, 8192);
  hipLaunchKernelGGL(add_inplace_kernel, dim3(grid), dim3(256), 0, st, x, r, n);
  return hipGetLastError();
}

// Segment i moves rows [src[i], src[i] + len[i]) of `from` to rows
// [dst[i], ...) of `to`, D floats per row; one grid-stride pass over all
// segments' float4s (segments never overlap).
__global__ void copy_rows_kernel(const float* __restrict__ from, float* __restrict__ to,
                                 RowCopyMap m, int D) {
  const int q = D / 4;
  const long total = (long)m.row_end[m.n - 1] * q;
  for (long i = blockIdx.x * 256L + threadIdx.x; i < total; i += (long)gridDim.x * 256) {
    const int row = (int)(i / q), c = (int)(i - (long)row * q);
    int s = 0;
#pragma unroll 1
    for (int k = 0; k + 1 < m.n; ++k) s += row >= m.row_end[k] ? 1 : 0;
    const int r = row - (s ? m.row_end[s - 1] : 0);
    ((float4*)to)[(long)(m.dst[s] + r) * q + c] = ((const float4*)from)[(long)(m.src[s] + r) * q + c];
  }
}

hipError_t launch_copy_rows(const float* from, float* to, const RowCopyMap& m, int D,
                            hipStream_t st) {
  if (m.n == 0) return hipSuccess;
  const long total = (long)m.row_end[m.n - 1] * (D / 4);
  if (total == 0) return hipSuccess;
  const int grid = (int)std::min<long>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(copy_rows_kernel, dim3(grid), dim3(256), 0, st, from, to, m, D);
  return hipGetLastError();
}

__global__ void bias_rows_f32_kernel(const bf16* __restrict__ b16, const float* __restrict__ b32,
                                     int rows, int D, float* __restrict__ dst) {
  const long n = (long)rows * D;
  for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
    const int d = (int)(i % D);
    dst[i] = b16 ? (float)b16[d] : b32[d];
  }
}

hipError_t launch_bias_rows_f32(const void* bias, bool bias_bf16, int rows, int D, float* dst,
                                hipStream_t st) {
  const long n = (long)rows * D;
  if (n == 0) return hipSuccess;
  const int grid = (int)std::min<long>((n + 255) / 256, 8192);
  hipLaunchKernelGGL(bias_rows_f32_kernel, dim3(grid), dim3(256), 0, st,
                     bias_bf16 ? (const bf16*)bias : nullptr,
                     bias_bf16 ? nullptr : (const float*)bias, rows, D, dst);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Final layer: per image token and guidance branch,
//   out = LNmod(x; shift, scale) W_out^T + b_out     (P = p*p*C outputs)
// then v = v_u + g (v_c - v_u), unpatchify, noise_pred = v, latent += dt v.
// One wave per token, both guidance branches together (each weight load
// serves both).  Each lane accumulates its share of every output (same
// per-lane FMA order as a per-output loop); for P a power of two the P sums
// are then finished by one butterfly reduce-scatter whose pairings are those
// of wave_sum, so every output is added up in exactly the same order.
template <typename TW, int PT>
__device__ __forceinline__ float4 ld_w4(const TW* w) {
  if constexpr (sizeof(TW) == 2) {
    const bf16x4 q = *(const bf16x4*)w;
    return float4{(float)q[0], (float)q[1], (float)q[2], (float)q[3]};
  } else {
    return *(const float4*)w;
  }
}

template <typename TW, int PT, int NV>
__global__ __launch_bounds__(256) void final_kernel(const float* __restrict__ x, ReqMap rm,
                                                    const TW* __restrict__ w_out,
                                                    const TW* __restrict__ b_out,
                                                    const float* __restrict__ mod, int ld_mod,
                                                    int shift_off, int scale_off, int D, int C,
                                                    int p, float eps, float guidance,
                                                    float* __restrict__ lat,
                                                    float* __restrict__ noise_pred) {
  constexpr int NI = NV ? (NV + 63) / 64 : kMaxV4;
  // DiT width 1152, 16 outputs, bf16: the workgroup's four waves read the
  // projection (36 KB) from LDS, staged once, instead of each from L2
  constexpr bool WLDS = PT == 16 && NV == 288 && sizeof(TW) == 2;
  __shared__ __attribute__((aligned(16))) TW wsh[WLDS ? 16 * 4 * 288 : 1];
  if constexpr (WLDS) {
    for (int i = threadIdx.x; i < 16 * 4 * 288 / 8; i += 256)
      ((bf16x8*)wsh)[i] = ((const bf16x8*)w_out)[i];
    __syncthreads();
  }
  const TW* wsrc = WLDS ? wsh : w_out;
  const int lane = threadIdx.x & 63;
  const int tok = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (tok >= rm.tokens_total) return;
  const int r = req_of_token(rm, tok);
  const int P = PT ? PT : p * p * C;
  const int nv = NV ? NV : D >> 2;
  const float* md = mod + (size_t)rm.modrow[r] * ld_mod;
  const float4* sh = (const float4*)(md + shift_off);
  const float4* sc = (const float4*)(md + scale_off);
  const int nb = rm.branches;
  float4 v[2][NI];
  // LN-modulate both branches' rows in registers (static indices throughout,
  // so that everything stays in registers)
#pragma unroll
  for (int br = 0; br < 2; ++br) {
    if (br >= nb) continue;
    const float4* xr = (const float4*)(x + ((size_t)br * rm.tokens_total + tok) * D);
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int c = lane + 64 * i;
      if (c < nv) {
        v[br][i] = xr[c];
        s += (v[br][i].x + v[br][i].y) + (v[br][i].z + v[br][i].w);
      }
    }
    const float mean = wave_sum(s) / (float)D;
    float q = 0.f;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int c = lane + 64 * i;
      if (c < nv) {
        const float a = v[br][i].x - mean, b = v[br][i].y - mean, cc = v[br][i].z - mean,
                    d = v[br][i].w - mean;
        q += (a * a + b * b) + (cc * cc + d * d);
      }
    }
    const float rstd = 1.0f / sqrtf(wave_sum(q) / (float)D + eps);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int c = lane + 64 * i;
      if (c < nv) {
        const float4 a = sh[c], b = sc[c];
        v[br][i].x = (v[br][i].x - mean) * rstd * (1.f + b.x) + a.x;
        v[br][i].y = (v[br][i].y - mean) * rstd * (1.f + b.y) + a.y;
        v[br][i].z = (v[br][i].z - mean) * rstd * (1.f + b.z) + a.z;
        v[br][i].w = (v[br][i].w - mean) * rstd * (1.f + b.w) + a.w;
      }
    }
  }
  float mine[2] = {0.f, 0.f};
  int f_own = lane;   // output this lane ends with
  if constexpr (PT > 0) {
    // per-lane partial sums of every output, then the reduce-scatter
    float acc[2][PT];
#pragma unroll
    for (int f = 0; f < PT; ++f) acc[0][f] = acc[1][f] = 0.f;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int c = lane + 64 * i;
      if (c < nv) {
#pragma unroll
        for (int f = 0; f < PT; ++f) {
          const float4 w = ld_w4<TW, PT>(wsrc + (size_t)f * D + 4 * c);
#pragma unroll
          for (int br = 0; br < 2; ++br) {
            acc[br][f] = fmaf(v[br][i].x, w.x, acc[br][f]);
            acc[br][f] = fmaf(v[br][i].y, w.y, acc[br][f]);
            acc[br][f] = fmaf(v[br][i].z, w.z, acc[br][f]);
            acc[br][f] = fmaf(v[br][i].w, w.w, acc[br][f]);
          }
        }
      }
    }
    // step st (lane bit o = 32 >> st) halves the outputs a lane holds -- it
    // keeps the half given by that bit -- until one is left, then plain
    // butterfly steps
    int base = 0;
#pragma unroll
    for (int st = 0; st < 6; ++st) {
      const int o = 32 >> st;
      const int K = PT >> st;          // outputs held before this step
      const bool up = (lane & o) != 0;
      if (K > 1) {
        const int h = K / 2;
#pragma unroll
        for (int br = 0; br < 2; ++br)
#pragma unroll
          for (int t = 0; t < h; ++t) {
            const float keep = up ? acc[br][t + h] : acc[br][t];
            const float send = up ? acc[br][t] : acc[br][t + h];
            acc[br][t] = keep + __shfl_xor(send, o, kWave);
          }
        if (up) base += h;
      } else {
#pragma unroll
        for (int br = 0; br < 2; ++br) acc[br][0] += __shfl_xor(acc[br][0], o, kWave);
      }
    }
    f_own = base;
    const float bo = to_f32(b_out[f_own]);
    mine[0] = acc[0][0] + bo;
    mine[1] = acc[1][0] + bo;
  } else {
#pragma unroll
    for (int br = 0; br < 2; ++br) {
      if (br >= nb) continue;
      for (int f = 0; f < P; ++f) {
        const TW* wr = w_out + (size_t)f * D;
        float part = 0.f;
#pragma unroll
        for (int i = 0; i < NI; ++i) {
          const int c = lane + 64 * i;
          if (c < nv) {
            part = fmaf(v[br][i].x, to_f32(wr[4 * c + 0]), part);
            part = fmaf(v[br][i].y, to_f32(wr[4 * c + 1]), part);
            part = fmaf(v[br][i].z, to_f32(wr[4 * c + 2]), part);
            part = fmaf(v[br][i].w, to_f32(wr[4 * c + 3]), part);
          }
        }
        const float tot = wave_sum(part) + to_f32(b_out[f]);
        if (lane == f) mine[br] = tot;
      }
    }
  }
  // one lane per output writes (for PT, the first of the lanes that hold it)
  if (PT > 0 ? (lane & (64 / (PT > 0 ? PT : 64) - 1)) != 0 : lane >= P) return;
  const float vel = nb == 2 ? mine[1] + guidance * (mine[0] - mine[1]) : mine[0];
  const int f = f_own;
  const int a = f / (p * C), b = (f / C) % p, c = f % C;
  const int lt = tok - rm.tok_off[r];
  const int W = rm.w[r], H = rm.h[r], gw = W / p;
  const int gi = lt / gw, gj = lt - gi * gw;
  const size_t li = (size_t)rm.lat_off[r] + (size_t)c * H * W + (size_t)(gi * p + a) * W + gj * p + b;
  if (noise_pred) noise_pred[li] = vel;
  const float dt = rm.dt[r];
  if (dt != 0.f) lat[li] = lat[li] + dt * vel;
}

// Final layer of the wide model (64 outputs of width 3072, bf16 weights):
// a workgroup takes kFwTok tokens so that each 64-column chunk of the
// projection, staged in LDS as fp32, serves all of them (the per-token wave
// above reads the 384 KB projection from L2 once per token).  Per guidance
// branch: the tokens' LayerNorm statistics (two passes over each row, one
// wave per token), then for each 64-column chunk the modulated rows and the
// projection's columns go to LDS and every thread accumulates 4 tokens x 2
// outputs in fp32, K ascending; then guidance, unpatchify, noise_pred and
// the Euler update as in final_kernel.
constexpr int kFwTok = 32, kFwK = 64, kFwP = 64;

__global__ __launch_bounds__(256) void final_wide_kernel(const float* __restrict__ x, ReqMap rm,
                                                         const bf16* __restrict__ w_out,
                                                         const bf16* __restrict__ b_out,
                                                         const float* __restrict__ mod, int ld_mod,
                                                         int shift_off, int scale_off, int D, int C,
                                                         int p, float eps, float guidance,
                                                         float* __restrict__ lat,
                                                         float* __restrict__ noise_pred) {
  __shared__ float hs[kFwTok][kFwK + 1];
  __shared__ float ws[kFwP][kFwK + 1];
  __shared__ float st_mean[kFwTok], st_rstd[kFwTok];
  __shared__ int st_row[kFwTok];   // modulation row of each token (-1 past the end)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int tok0 = blockIdx.x * kFwTok;
  const int T = rm.tokens_total, nb = rm.branches;
  const int ty = tid >> 5, tx = tid & 31;   // tokens 4 ty .. +3, outputs 2 tx, 2 tx + 1
  if (tid < kFwTok) {
    const int t = tok0 + tid;
    st_row[tid] = t < T ? rm.modrow[req_of_token(rm, t)] : -1;
  }
  float res[2][4][2];
#pragma unroll
  for (int br = 0; br < 2; ++br) {
    if (br >= nb) break;
    __syncthreads();
    // statistics: wave w takes tokens w, w + 4, ...
    for (int i = wave; i < kFwTok; i += 4) {
      const int t = tok0 + i;
      float mean = 0.f, rstd = 0.f;
      if (t < T) {
        const float4* xr = (const float4*)(x + ((size_t)br * T + t) * D);
        float s = 0.f;
        for (int c = lane; c < D / 4; c += 64) {
          const float4 v = xr[c];
          s += (v.x + v.y) + (v.z + v.w);
        }
        mean = wave_sum(s) / (float)D;
        float q = 0.f;
        for (int c = lane; c < D / 4; c += 64) {
          const float4 v = xr[c];
          const float a = v.x - mean, b = v.y - mean, cc = v.z - mean, d = v.w - mean;
          q += (a * a + b * b) + (cc * cc + d * d);
        }
        rstd = 1.0f / sqrtf(wave_sum(q) / (float)D + eps);
      }
      if (lane == 0) {
        st_mean[i] = mean;
        st_rstd[i] = rstd;
      }
    }
    float acc[4][2] = {{0.f, 0.f}, {0.f, 0.f}, {0.f, 0.f}, {0.f, 0.f}};
    for (int k0 = 0; k0 < D; k0 += kFwK) {
      __syncthreads();
      // modulated rows: 32 tokens x 64 columns, 8 per thread (2 float4)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int e = tid + 256 * j, t = e >> 4, c4 = (e & 15) * 4;
        float4 h = float4{0.f, 0.f, 0.f, 0.f};
        const int mr = st_row[t];
        if (mr >= 0) {
          const float4 v = *(const float4*)(x + ((size_t)br * T + tok0 + t) * D + k0 + c4);
          const float* md = mod + (size_t)mr * ld_mod;
          const float4 sh = *(const float4*)(md + shift_off + k0 + c4);
          const float4 sc = *(const float4*)(md + scale_off + k0 + c4);
          const float mu = st_mean[t], rs = st_rstd[t];
          h.x = (v.x - mu) * rs * (1.f + sc.x) + sh.x;
          h.y = (v.y - mu) * rs * (1.f + sc.y) + sh.y;
          h.z = (v.z - mu) * rs * (1.f + sc.z) + sh.z;
          h.w = (v.w - mu) * rs * (1.f + sc.w) + sh.w;
        }
        hs[t][c4] = h.x;
        hs[t][c4 + 1] = h.y;
        hs[t][c4 + 2] = h.z;
        hs[t][c4 + 3] = h.w;
      }
      // the projection's 64 x 64 chunk, 16 per thread (2 x 8 bf16)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int e = tid + 256 * j, f = e >> 3, c8 = (e & 7) * 8;
        const bf16x8 w = *(const bf16x8*)(w_out + (size_t)f * D + k0 + c8);
#pragma unroll
        for (int q = 0; q < 8; ++q) ws[f][c8 + q] = (float)w[q];
      }
      __syncthreads();
#pragma unroll 8
      for (int k = 0; k < kFwK; ++k) {
        const float w0 = ws[2 * tx][k], w1 = ws[2 * tx + 1][k];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float h = hs[4 * ty + i][k];
          acc[i][0] = fmaf(h, w0, acc[i][0]);
          acc[i][1] = fmaf(h, w1, acc[i][1]);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      res[br][i][0] = acc[i][0];
      res[br][i][1] = acc[i][1];
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int tok = tok0 + 4 * ty + i;
    if (tok >= T) continue;
    const int r = req_of_token(rm, tok);
    const int lt = tok - rm.tok_off[r];
    const int W = rm.w[r], H = rm.h[r], gw = W / p;
    const int gi = lt / gw, gj = lt - gi * gw;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int f = 2 * tx + j;
      const float bo = (float)b_out[f];
      const float vc = res[0][i][j] + bo;
      const float vel = nb == 2 ? (res[1][i][j] + bo) + guidance * (vc - (res[1][i][j] + bo)) : vc;
      const int a = f / (p * C), b = (f / C) % p, c = f % C;
      const size_t li =
          (size_t)rm.lat_off[r] + (size_t)c * H * W + (size_t)(gi * p + a) * W + gj * p + b;
      if (noise_pred) noise_pred[li] = vel;
      const float dt = rm.dt[r];
      if (dt != 0.f) lat[li] = lat[li] + dt * vel;
    }
  }
}

hipError_t launch_final_layer(const float* x, const ReqMap& rm, const void* w_out,
                              const void* b_out, bool w_bf16, const float* mod, int ld_mod,
                              int shift_off, int scale_off, int D, int C, int p, float eps,
                              float guidance, float* latents, float* noise_pred, hipStream_t st) {
  if (rm.tokens_total == 0) return hipSuccess;
  dim3 grid((rm.tokens_total + 3) / 4), block(256);
  const int P = p * p * C;
#define T2I_FIN(TW_, PT_, NV_)                                                                 \
  hipLaunchKernelGGL((final_kernel<TW_, PT_, NV_>), grid, block, 0, st, x, rm, (const TW_*)w_out, \
                     (const TW_*)b_out, mod, ld_mod, shift_off, scale_off, D, C, p, eps, guidance, \
                     latents, noise_pred)
  if (w_bf16) {
    if (P == 16 && D == 1152) T2I_FIN(bf16, 16, 288);
    else if (P == kFwP && D % kFwK == 0 && (uintptr_t)w_out % 16 == 0) {
      hipLaunchKernelGGL(final_wide_kernel, dim3((rm.tokens_total + kFwTok - 1) / kFwTok), block,
                         0, st, x, rm, (const bf16*)w_out, (const bf16*)b_out, mod, ld_mod,
                         shift_off, scale_off, D, C, p, eps, guidance, latents, noise_pred);
      return hipGetLastError();
    }
    else if (P == 16) T2I_FIN(bf16, 16, 0);
    else T2I_FIN(bf16, 0, 0);
  } else {
    if (P == 16) T2I_FIN(float, 16, 0);
    else T2I_FIN(float, 0, 0);
  }
#undef T2I_FIN
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Step-skip cache.
//
// cache_signal_kernel: workgroup = 16 rows of one request.  m = LNmod(x0;
// block-0 shift_msa, scale_msa) in fp32; partial[blk] = (sum|m - m_prev|,
// sum|m_prev|) in fp64 (lane order, butterfly, then waves 0..3); m_prev := m.
// cache_decide_kernel: one thread per request sums its partials in block
// order and applies the rule.

int cache_partial_blocks(const ReqMap& rm) {
  int n = 0;
  for (int r = 0; r < rm.n; ++r)
    n += (rm.tok_off[r + 1] - rm.tok_off[r] + kCacheRowsPerBlock - 1) / kCacheRowsPerBlock;
  return n;
}

__global__ __launch_bounds__(256) void cache_signal_kernel(
    const float* __restrict__ x0, ReqMap rm, const float* __restrict__ mod, int ld_mod,
    int shift_off, int scale_off, int D, float eps, float* __restrict__ m_prev,
    const CacheHeader* __restrict__ hdr, int step, double* __restrict__ partial) {
  __shared__ double red[4][2];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // block -> (request, row chunk)
  int r = 0, base = 0;
  for (;;) {
    const int nb = (rm.tok_off[r + 1] - rm.tok_off[r] + kCacheRowsPerBlock - 1) / kCacheRowsPerBlock;
    if ((int)blockIdx.x < base + nb || r == rm.n - 1) break;
    base += nb;
    ++r;
  }
  const int chunk = blockIdx.x - base;
  const bool have_prev = step > 0 && hdr[r].has_m;
  const float* md = mod + (size_t)rm.modrow[r] * ld_mod;
  const float4* sh = (const float4*)(md + shift_off);
  const float4* sc = (const float4*)(md + scale_off);
  const int nv = D >> 2;
  double num = 0.0, den = 0.0;
  for (int rr = 0; rr < kCacheRowsPerBlock / 4; ++rr) {
    const int tok = rm.tok_off[r] + chunk * kCacheRowsPerBlock + wave * (kCacheRowsPerBlock / 4) + rr;
    if (tok >= rm.tok_off[r + 1]) break;
    const float4* xr = (const float4*)(x0 + (size_t)tok * D);
    float4* mr = (float4*)(m_prev + (size_t)tok * D);
    float4 v[kMaxV4];
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxV4; ++i) {
      const int c = lane + 64 * i;
      if (c < nv) {
        v[i] = xr[c];
        s += (v[i].x + v[i].y) + (v[i].z + v[i].w);
      }
    }
    const float mean = wave_sum(s) / (float)D;
    float q = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxV4; ++i) {
      const int c = lane + 64 * i;
      if (c < nv) {
        const float a = v[i].x - mean, b = v[i].y - mean, cc = v[i].z - mean, d = v[i].w - mean;
        q += (a * a + b * b) + (cc * cc + d * d);
      }
    }
    const float rstd = 1.0f / sqrtf(wave_sum(q) / (float)D + eps);
#pragma unroll
    for (int i = 0; i < kMaxV4; ++i) {
      const int c = lane + 64 * i;
      if (c < nv) {
        const float4 a = sh[c], b = sc[c];
        float4 m;
        m.x = (v[i].x - mean) * rstd * (1.f + b.x) + a.x;
        m.y = (v[i].y - mean) * rstd * (1.f + b.y) + a.y;
        m.z = (v[i].z - mean) * rstd * (1.f + b.z) + a.z;
        m.w = (v[i].w - mean) * rstd * (1.f + b.w) + a.w;
        if (have_prev) {
          const float4 o = mr[c];
          num += (double)fabsf(m.x - o.x) + (double)fabsf(m.y - o.y) +
                 (double)fabsf(m.z - o.z) + (double)fabsf(m.w - o.w);
          den += (double)fabsf(o.x) + (double)fabsf(o.y) + (double)fabsf(o.z) + (double)fabsf(o.w);
        }
        mr[c] = m;
      }
    }
  }
  num = wave_sum(num);
  den = wave_sum(den);
  if (lane == 0) {
    red[wave][0] = num;
    red[wave][1] = den;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    partial[2 * blockIdx.x + 0] = ((red[0][0] + red[1][0]) + red[2][0]) + red[3][0];
    partial[2 * blockIdx.x + 1] = ((red[0][1] + red[1][1]) + red[2][1]) + red[3][1];
  }
}

__global__ void cache_decide_kernel(ReqMap rm, const double* __restrict__ partial,
                                    CacheHeader* __restrict__ hdr, int step, int n_steps,
                                    double tau, int mode) {
  const int r = threadIdx.x;
  if (r >= rm.n) return;
  int b0 = 0;
  for (int i = 0; i < r; ++i)
    b0 += (rm.tok_off[i + 1] - rm.tok_off[i] + kCacheRowsPerBlock - 1) / kCacheRowsPerBlock;
  const int nb = (rm.tok_off[r + 1] - rm.tok_off[r] + kCacheRowsPerBlock - 1) / kCacheRowsPerBlock;
  CacheHeader hd = hdr[r];
  if (step == 0) {
    hd.acc = 0.0;
    hd.has_m = 0;
    hd.has_r = 0;
  }
  double d = __longlong_as_double(0x7ff8000000000000LL);   // NaN: no predecessor
  if (hd.has_m) {
    double num = 0.0, den = 0.0;
    for (int b = 0; b < nb; ++b) {
      num += partial[2 * (b0 + b) + 0];
      den += partial[2 * (b0 + b) + 1];
    }
    d = num / den;
  }
  int skip = 0;
  double acc = hd.acc;
  if (tau > 0.0 && step != 0 && step != n_steps - 1 && hd.has_r && hd.has_m) {
    if (mode == 0) {
      acc = acc + d;
      skip = acc < tau;
    } else {
      acc = d;
      skip = d < tau;
    }
  }
  if (!skip) acc = 0.0;
  hd.acc = acc;
  hd.d = d;
  hd.skip = skip;
  hd.has_m = 1;
  hdr[r] = hd;
}

hipError_t launch_cache_signal(const float* x0, const ReqMap& rm, const float* mod, int ld_mod,
                               int shift_off, int scale_off, int D, float eps, float* m_prev,
                               CacheHeader* hdr, int step, double* partial, hipStream_t st) {
  const int nb = cache_partial_blocks(rm);
  if (nb == 0) return hipSuccess;
  hipLaunchKernelGGL(cache_signal_kernel, dim3(nb), dim3(256), 0, st, x0, rm, mod, ld_mod,
                     shift_off, scale_off, D, eps, m_prev, hdr, step, partial);
  return hipGetLastError();
}

hipError_t launch_cache_decide(const ReqMap& rm, const double* partial, CacheHeader* hdr,
                               int step, int n_steps, double tau, int mode, hipStream_t st) {
  hipLaunchKernelGGL(cache_decide_kernel, dim3(1), dim3(64), 0, st, rm, partial, hdr, step,
                     n_steps, tau, mode);
  return hipGetLastError();
}

// x[b][tok] = x0[tok] + R[b][tok] (skip_mask) / R[b][tok] = x[b][tok] - x0[tok] (store_mask)
__global__ void residual_kernel(const float* __restrict__ x0, const float* __restrict__ R_in,
                                float* __restrict__ x, float* __restrict__ R_out, ReqMap rm,
                                uint32_t mask, int D, int store, CacheHeader* __restrict__ hdr) {
  const int nv = D >> 2;
  const long per_branch = (long)rm.tokens_total * nv;
  const long total = per_branch * rm.branches;
  if (store && blockIdx.x == 0 && threadIdx.x < (unsigned)rm.n && ((mask >> threadIdx.x) & 1u))
    hdr[threadIdx.x].has_r = 1;
  for (long i = blockIdx.x * 256L + threadIdx.x; i < total; i += (long)gridDim.x * 256) {
    const int br = (int)(i / per_branch);
    const long j = i - (long)br * per_branch;
    const int tok = (int)(j / nv);
    const int r = req_of_token(rm, tok);
    if (!((mask >> r) & 1u)) continue;
    const float4 a = ((const float4*)x0)[j];
    if (store) {
      const float4 b = ((const float4*)x)[i];
      ((float4*)R_out)[i] = float4{b.x - a.x, b.y - a.y, b.z - a.z, b.w - a.w};
    } else {
      const float4 b = ((const float4*)R_in)[i];
      ((float4*)x)[i] = float4{a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w};
    }
  }
}

hipError_t launch_apply_residual(const float* x0, const float* R, float* x, const ReqMap& rm,
                                 uint32_t skip_mask, int D, hipStream_t st) {
  const long total = (long)rm.tokens_total * (D / 4) * rm.branches;
  if (total == 0 || skip_mask == 0) return hipSuccess;
  const int grid = (int)std::min<long>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(residual_kernel, dim3(grid), dim3(256), 0, st, x0, R, x, (float*)nullptr, rm,
                     skip_mask, D, 0, (CacheHeader*)nullptr);
  return hipGetLastError();
}

hipError_t launch_store_residual(const float* x0, const float* x, float* R, const ReqMap& rm,
                                 uint32_t store_mask, int D, CacheHeader* hdr, hipStream_t st) {
  const long total = (long)rm.tokens_total * (D / 4) * rm.branches;
  if (total == 0 || store_mask == 0) return hipSuccess;
  const int grid = (int)std::min<long>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(residual_kernel, dim3(grid), dim3(256), 0, st, x0, (const float*)nullptr,
                     (float*)x, R, rm, store_mask, D, 1, hdr);
  return hipGetLastError();
}

}  // namespace t2i
