// Internal declarations shared by the gfx950 kernels and the host orchestration.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace t2i {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kMaxSeq = 64;
constexpr int kMaxReq = 32;
constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Small tables passed to kernels by value (no device copies, no memcpy).

// Packed rows -> sequence.  Sequence s owns rows [start[s], start[s+1]); its
// modulation-table row is modrow[s].
struct SeqMap {
  int n;
  int start[kMaxSeq + 1];
  int modrow[kMaxSeq];
};

// Variable-length attention: query sequence s reads Q rows [q_start, +q_len)
// and attends to the K/V rows [k_start, +k_len) followed by the optional
// second segment [k2_start, +k2_len) (joint attention: a request's text rows
// and its image rows live in different parts of the buffers).  tile_start[s]
// is the first query tile of s in the flattened tile space of one head
// (prefix sum of ceil(q_len/BQ)).
struct AttnMap {
  int n;
  int waves;   // 32-query waves per workgroup (bf16 kernel): the query tile is 32 * waves
  int q_start[kMaxSeq], q_len[kMaxSeq], k_start[kMaxSeq], k_len[kMaxSeq];
  int k2_start[kMaxSeq], k2_len[kMaxSeq];
  int tile_start[kMaxSeq + 1];
};

// Cross-attention fused into its query projection (gemm_dma_kernel with XAttnArgs): the
// query rows of sequence s are [q_start[s], +q_len[s]) (multiples of 256, so
// that a 256-row tile lies in one sequence); its text is K rows
// [k_start[s], +k_len[s]) (row-major, stride ldk, 1 .. 128 rows) and the
// same columns of V^T (stride ldvt); the attention output goes to O (stride
// ldo), the queries themselves are not stored.
struct XAttnArgs {
  static constexpr bool on = true;
  const bf16* K;
  int ldk;
  const bf16* Vt;
  int ldvt;
  bf16* O;
  int ldo;
  int n;
  int q_start[kMaxSeq], q_len[kMaxSeq], k_start[kMaxSeq], k_len[kMaxSeq];
};

// Per-request geometry for the image-side kernels.
struct ReqMap {
  int n;                    // requests
  int tokens_total;         // image tokens of all requests (one branch)
  int branches;             // 1 or 2
  int tok_off[kMaxReq + 1]; // first token of request r within a branch
  int lat_off[kMaxReq];     // first float of request r's latent
  int h[kMaxReq], w[kMaxReq];
  int modrow[kMaxReq];      // modulation-table row of request r
  float dt[kMaxReq];        // Euler step t_next - t (0 = no update)
};

// Timestep values handed to a kernel by value (host array, no copy).
constexpr int kTValsChunk = 64;
struct TVals {
  int n;
  double t[kTValsChunk];
};

__device__ __forceinline__ int seq_of_row(const SeqMap& m, int row) {
  int s = 0;
  #pragma unroll 1
  for (int i = 1; i < m.n; ++i) s += (row >= m.start[i]) ? 1 : 0;
  return s;
}

__device__ __forceinline__ int req_of_token(const ReqMap& m, int tok) {
  int r = 0;
  #pragma unroll 1
  for (int i = 1; i < m.n; ++i) r += (tok >= m.tok_off[i]) ? 1 : 0;
  return r;
}

// ---------------------------------------------------------------------------
// Conversions and reductions.

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16 v) { return (float)v; }
template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) { return (bf16)v; }

__device__ __forceinline__ float wave_sum(float v) {
  #pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ double wave_sum(double v) {
  #pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// GELU with the tanh approximation, written as u * sigmoid(2z):
// 0.5 u (1 + tanh z) = u / (1 + exp(-2z)),  z = sqrt(2/pi) (u + 0.044715 u^3).
// The reciprocal is the hardware v_rcp_f32 (about 1 ulp), not an IEEE
// division: exp(-2z) -> +inf gives rcp(inf) = 0 and u * 0 = -0 for u -> -inf,
// matching the limit.
// u * sigmoid(2 z), z = sqrt(2/pi) (u + 0.044715 u^3): exp(-2 z) taken as
// 2^(u (c1 + c2 u^2)) with the constants folded (one multiply-add and two
// multiplies before the exponential)
__device__ __forceinline__ float gelu_tanh(float u) {
  constexpr float c1 = -2.0f * 0.7978845608028654f * 1.4426950408889634f;
  constexpr float c2 = c1 * 0.044715f;
  const float t = u * fmaf(c2, u * u, c1);
  return u * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(t));
}

__device__ __forceinline__ float silu(float v) { return v * __builtin_amdgcn_rcpf(1.0f + __expf(-v)); }

// ---------------------------------------------------------------------------
// Linear-layer epilogue.

enum EpiKind { EPI_STORE = 0, EPI_GELU = 1, EPI_SILU = 2, EPI_RESID = 3, EPI_RESID_GATED = 4,
               EPI_SPLIT_VT = 5, EPI_STORE_F32 = 6,
               EPI_PARTIAL = 7 /* split-K partial sums, fp32, no bias */ };

struct Epi {
  void* out;          // STORE / GELU / SILU destination (SPLIT_VT: columns < vcol0)
  int ldo;
  bf16* vt;           // SPLIT_VT: columns >= vcol0 stored transposed, vt[(n - vcol0) * ldvt + m]
  int ldvt;
  int vcol0;
  float* x;           // fp32 residual for RESID kinds
  int ldx;
  bf16* xb;           // optional bf16 copy of the updated residual (stride ldx)
  const float* gate;  // gate rows: gate[modrow(seq(row)) * ld_gate + col]
  int ld_gate;
  SeqMap map;
  // STORE / SPLIT_VT: columns < qcols (a multiple of 4) are multiplied by
  // qscale before their one rounding to bf16 -- the attention queries,
  // written already scaled by log2(e)/sqrt(d) (0 = no column scaled)
  float qscale;
  int qcols;
};

template <typename OutT>
__device__ __forceinline__ void epi_apply(const Epi& e, int kind, int m, int n, float y) {
  if (kind == EPI_STORE) {
    if (n < e.qcols) y *= e.qscale;
    ((OutT*)e.out)[(size_t)m * e.ldo + n] = from_f32<OutT>(y);
  } else if (kind == EPI_STORE_F32) {
    ((float*)e.out)[(size_t)m * e.ldo + n] = y;
  } else if (kind == EPI_SPLIT_VT) {
    if (n < e.qcols) y *= e.qscale;
    if (n < e.vcol0) ((OutT*)e.out)[(size_t)m * e.ldo + n] = from_f32<OutT>(y);
    else e.vt[(size_t)(n - e.vcol0) * e.ldvt + m] = (bf16)y;
  } else if (kind == EPI_GELU) {
    ((OutT*)e.out)[(size_t)m * e.ldo + n] = from_f32<OutT>(gelu_tanh(y));
  } else if (kind == EPI_SILU) {
    ((OutT*)e.out)[(size_t)m * e.ldo + n] = from_f32<OutT>(silu(y));
  } else {
    float g = 1.0f;
    if (kind == EPI_RESID_GATED) {
      int s = seq_of_row(e.map, m);
      g = e.gate[(size_t)e.map.modrow[s] * e.ld_gate + n];
    }
    size_t i = (size_t)m * e.ldx + n;
    float nx = e.x[i] + g * y;
    e.x[i] = nx;
    if (e.xb) e.xb[i] = (bf16)nx;
  }
}

// ---------------------------------------------------------------------------
// Launchers (defined in the kernel files; all asynchronous on `st`).

// splitk_ws (fp32, splitk_floats of room, or NULL): lets a short-M, long-K
// layer split K over several workgroups (partial sums there, then a
// fixed-order reduction that applies the epilogue)
hipError_t launch_gemm_bf16(const bf16* A, int lda, const bf16* W, int ldw, const bf16* bias,
                            int M, int N, int K, int kind, const Epi& epi, float* splitk_ws,
                            size_t splitk_floats, hipStream_t st);

// SIMT fp32-accumulating GEMM: A fp32, W fp32 or bf16 (w_bf16), bias like W,
// output fp32 for STORE kinds.
hipError_t launch_gemm_f32(const float* A, int lda, const void* W, int ldw, bool w_bf16,
                           const void* bias, int M, int N, int K, int kind, const Epi& epi,
                           hipStream_t st);

// Conditioning GEMMs: A fp32 [M, K], W fp32 or bf16 [N, K]; STORE or SILU.
// Per-group operand table of a grouped launch (by value in the kernel
// arguments): group i uses W[i], bias[i] and writes out[i] (vt[i]).
constexpr int kMaxGroups = 64;
struct PtrGroup {
  const void* W[kMaxGroups];
  const void* bias[kMaxGroups];
  void* out[kMaxGroups];
  bf16* vt[kMaxGroups];
};

// Grouped bf16 GEMM over shapes that launch_gemm_bf16 runs on its
// register-staged tiles without split-K (gemm_bf16_groupable); STORE or
// SPLIT_VT epilogue; bitwise the per-group launch_gemm_bf16 results.
bool gemm_bf16_groupable(int M, int N, int kind);
hipError_t launch_gemm_bf16_group(const bf16* A, int lda, const PtrGroup& g, int groups, int ldw,
                                  int M, int N, int K, int kind, const Epi& epi, hipStream_t st);
// Grouped conditioning GEMV (EPI_STORE), bitwise the per-group
// launch_linear_rows results.
hipError_t launch_linear_rows_group(const float* A, int lda, const PtrGroup& g, int groups,
                                    int ldw, bool w_bf16, int M, int N, int K, const Epi& epi,
                                    hipStream_t st);
hipError_t launch_linear_rows(const float* A, int lda, const void* W, int ldw, bool w_bf16,
                              const void* bias, int M, int N, int K, int kind, const Epi& epi,
                              hipStream_t st);

// role: 0 self / joint attention, 1 cross-attention (same kernel, own instance).
// q_prescaled (bf16 only): Q was written multiplied by log2(e)/sqrt(head_dim)
// (Epi::qscale), so scores come out of the MFMA in log2 units; otherwise the
// kernel applies that scale to each score in fp32.
// The cross-attention query projection (epi: EPI_STORE's query scaling)
// followed in the same kernel by the cross-attention of xa; the queries are
// not stored.  hipErrorNotSupported (nothing launched) where the shapes do
// not fit the fused kernel; check_only: only those checks.
hipError_t launch_gemm_xattn(const bf16* A, int lda, const bf16* W, int ldw, const bf16* bias,
                             int M, int N, int K, const Epi& epi, int heads, int head_dim,
                             const XAttnArgs& xa, hipStream_t st, bool check_only = false);
hipError_t launch_attention(bool bf16_io, int role, int heads, int head_dim, const AttnMap& map,
                            const void* q, int ldq, const void* k, int ldk, const void* v,
                            int ldv, void* o, int ldo, hipStream_t st, bool q_prescaled);
// log2(e) / sqrt(head_dim): the query scale of q_prescaled attention
inline float attn_q_scale(int head_dim) {
  return 1.4426950408889634f / __builtin_sqrtf((float)head_dim);
}
// Query tiling of a map whose q_len are set: chooses the waves per workgroup
// (fewer, smaller workgroups when the default tiling would not fill the
// chip) and fills waves and tile_start.  Every 32-query group is computed
// the same way whatever the tiling.
void attention_tiles(AttnMap& m, bool bf16_io, int heads, int role);

hipError_t launch_ln_modulate(bool bf16_out, int rows, int D, const float* x, int ldx,
                              const float* mod, int ld_mod, int shift_off, int scale_off,
                              const SeqMap& map, void* out, int ldo, float eps, hipStream_t st);

// pe_table: workspace for the 2D sin-cos table (pe_npos x D/4 float2), NULL
// for no position embedding; pe_npos = largest grid side of the call
hipError_t launch_embed(const float* lat, const ReqMap& rm, const void* w_pe, const void* b_pe,
                        bool w_bf16, int D, int C, int p, float2* pe_table, int pe_npos,
                        float* x0, float* x, int copies, hipStream_t st);

// t: HOST array of `rows` timesteps (launched in chunks of kTValsChunk).
hipError_t launch_timestep_freq(const double* t, int rows, int freq_dim, double t_scale,
                                float* out, hipStream_t st);

hipError_t launch_broadcast_rows(const void* src, bool bf16_io, int rows, int D, void* dst,
                                 hipStream_t st);

hipError_t launch_final_layer(const float* x, const ReqMap& rm, const void* w_out,
                              const void* b_out, bool w_bf16, const float* mod, int ld_mod,
                              int shift_off, int scale_off, int D, int C, int p, float eps,
                              float guidance, float* latents, float* noise_pred, hipStream_t st);

// 2D RoPE.  table[pos * q + j] = (cos, sin)(pos * 10000^(-j/q)), q = head_dim/4,
// pos < npos; rope_apply rotates, in place, the q (columns [0, D)) and k
// (columns [D, 2D)) of the image rows [row0, row0 + branches * tokens) of a
// bf16 buffer with row stride ld: the first head_dim/2 dims of each head by
// the token's grid row, the last head_dim/2 by its grid column, pairs (2j, 2j+1).
hipError_t launch_rope_table(float2* table, int npos, int q, hipStream_t st);
hipError_t launch_rope_apply(bf16* qk, int ld, int row0, const ReqMap& rm, int heads, int head_dim,
                             int patch, const float2* table, hipStream_t st);
// W <- W + alpha B A (LoRA merge), W [n_out, n_in] stride ldw, rank <= 128
// the same merge for n <= kMaxGroups weights of one shape, weight i from
// W[i] (stride ldw) with A[i], B[i]: one launch
struct LoraGroup {
  void* W[kMaxGroups];
  const void* A[kMaxGroups];
  const void* B[kMaxGroups];
};
hipError_t launch_lora_merge_group(bool bf16_io, int n, int n_out, int n_in, int rank,
                                   float alpha, const LoraGroup& g, int ldw, hipStream_t st);
hipError_t launch_lora_merge(bool bf16_io, int n_out, int n_in, int rank, float alpha, void* W,
                             int ldw, const void* A, const void* B, hipStream_t st);
// Row segments to move between two fp32 [rows, D] buffers: segment i takes
// rows src[i] .. of the source to rows dst[i] .. of the destination; row_end
// is the running total of segment lengths (segment i has row_end[i] -
// row_end[i-1] rows).  D % 4 == 0.
struct RowCopyMap {
  int n;
  int src[kMaxSeq], dst[kMaxSeq], row_end[kMaxSeq];
};
hipError_t launch_copy_rows(const float* from, float* to, const RowCopyMap& m, int D,
                            hipStream_t st);
// Reads bytes (a multiple of 1024, below 2 GiB) of src once through the
// direct-to-LDS load path; writes kDmaReadGroups floats to sink.
constexpr int kDmaReadGroups = 1024;
hipError_t launch_dma_read(const void* src, size_t bytes, float* sink, hipStream_t st);
// x[i] += r[i] for i < n (fp32)
hipError_t launch_add_inplace(float* x, const float* r, size_t n, hipStream_t st);
// dst[r][:] = float(bias[:]) for r < rows (bf16 or fp32 bias)
hipError_t launch_bias_rows_f32(const void* bias, bool bias_bf16, int rows, int D, float* dst,
                                hipStream_t st);

// Cache-skip support.
struct CacheHeader {      // one per request, in the caller's cache-state buffer
  double acc;             // accumulated relative L1 change
  double d;               // last d_k
  int32_t has_m;          // m_prev valid
  int32_t has_r;          // residual valid
  int32_t skip;           // last decision
  int32_t pad;
};
constexpr int kCacheRowsPerBlock = 16;

int cache_partial_blocks(const ReqMap& rm);
hipError_t launch_cache_signal(const float* x0, const ReqMap& rm, const float* mod, int ld_mod,
                               int shift_off, int scale_off, int D, float eps, float* m_prev,
                               CacheHeader* hdr, int step, double* partial, hipStream_t st);
hipError_t launch_cache_decide(const ReqMap& rm, const double* partial, CacheHeader* hdr,
                               int step, int n_steps, double tau, int mode, hipStream_t st);
// x[b][tok] = x0[tok] + R[b][tok] for requests with skip_mask[r]
hipError_t launch_apply_residual(const float* x0, const float* R, float* x, const ReqMap& rm,
                                 uint32_t skip_mask, int D, hipStream_t st);
// R[b][tok] = x[b][tok] - x0[tok] for requests with store_mask[r]; sets has_r
hipError_t launch_store_residual(const float* x0, const float* x, float* R, const ReqMap& rm,
                                 uint32_t store_mask, int D, CacheHeader* hdr, hipStream_t st);

}  // namespace t2i
