/*
 * t2i_ops.h -- kernel-level entry points of the denoising step.
 *
 * The same kernels t2i_dit_step launches, exposed one by one so that each can
 * be checked against its definition in isolation.  Conventions are those of
 * t2i_dit.h: device pointers are caller-owned HIP memory, `stream` is a
 * hipStream_t as void*, launches are asynchronous, arguments are validated
 * before any launch, errors come back as t2i_status (text in
 * t2i_ops_last_error(), per host thread).
 */
#ifndef T2I_OPS_H
#define T2I_OPS_H

#include <stdint.h>
#include "t2i_dit.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Epilogues of the linear layer y = A W^T + b. */
typedef enum {
  T2I_EPI_STORE = 0,       /* out = y */
  T2I_EPI_GELU = 1,        /* out = GELU_tanh(y) */
  T2I_EPI_SILU = 2,        /* out = SiLU(y) */
  T2I_EPI_RESID = 3,       /* resid += y  (fp32), resid_copy = bf16(resid) */
  T2I_EPI_RESID_GATED = 4  /* resid += gate (.) y, gate a [N] fp32 vector */
} t2i_epilogue;

/*
 * Linear layer (DiT projections, Sec. 4's model `forward`): y = A W^T + b,
 * A [M, K] with row stride lda, W [N, K] with row stride ldw, b [N].
 *   dtype T2I_BF16: A, W, b bf16, MFMA with fp32 accumulation, K % 64 == 0,
 *                   lda, ldw % 8 == 0.  `out` is bf16.
 *   dtype T2I_F32 : A, W, b, out fp32.
 * For T2I_EPI_RESID*: `resid` is fp32 [M, N] (stride ldr) updated in place,
 * `resid_copy` (bf16 [M, N], stride ldr, or NULL) receives its new value;
 * `out` is unused.  `gate` is fp32 [N] (T2I_EPI_RESID_GATED only).
 */
t2i_status t2i_op_linear(int32_t dtype, int32_t epilogue, int32_t M, int32_t N,
                         int32_t K, const void* A, int32_t lda, const void* W,
                         int32_t ldw, const void* bias, void* out, int32_t ldo,
                         float* resid, int32_t ldr, void* resid_copy,
                         const float* gate, void* stream);

/*
 * Multi-head attention softmax(Q K^T / sqrt(d)) V over packed variable-length
 * sequences (the DiT's self- and cross-attention, Sec. 4's model `forward`;
 * joint text+image attention of the Sec. 8.1 model family): query sequence s
 * holds rows q_start[s] .. q_start[s]+q_len[s]-1 of Q and attends to rows
 * k_start[s] .. +k_len[s]-1 of K and V and, when k2_start/k2_len are given
 * (both or neither), also to rows k2_start[s] .. +k2_len[s]-1 -- the joint
 * attention's text keys and image keys, wherever each stream's rows sit.
 * Host arrays of n_seq <= T2I_MAX_SEQ entries; k_len + k2_len >= 1.  Head h of
 * a row occupies columns h*d .. h*d+d-1.  Q, K, O are dtype (bf16 or fp32)
 * with row strides ldq, ldk, ldo (multiples of 8).
 *   fp32: V is row-major like K, row stride ldv.
 *   bf16: V is given transposed, V^T [heads*head_dim][ldv] (the key index is
 *         contiguous), the layout the fused qkv projection writes; every key
 *         segment must start at a multiple of 8 and end within ldv.  The
 *         kernel addresses K and V^T with 32-bit byte offsets:
 *         2*heads*head_dim*ldv and 2*(last key row + 64)*ldk must stay below
 *         2^31, else T2I_ERR_SHAPE.
 */
t2i_status t2i_op_attention(int32_t dtype, int32_t heads, int32_t head_dim,
                            int32_t n_seq, const int32_t* q_start,
                            const int32_t* q_len, const int32_t* k_start,
                            const int32_t* k_len, const int32_t* k2_start,
                            const int32_t* k2_len, const void* q, int32_t ldq,
                            const void* k, int32_t ldk, const void* v,
                            int32_t ldv, void* o, int32_t ldo, void* stream);

/*
 * Cross-attention of image queries to their request's text (Sec. 4's model
 * `forward`, the DiT block's attention to the caption): the operation of
 * t2i_op_attention with one key segment per sequence, bf16 only (else
 * T2I_ERR_INVALID_ARG), run by the kernels the model uses for it where it
 * does not fuse it into the query projection (t2i_op_linear_cross_attention)
 * -- texts of at most 128 keys (k_len 1..128) by the two-tile kernel that
 * keeps them in LDS across query tiles, longer texts by the pipelined one.
 * Arguments, layouts (V given transposed) and limits are those of
 * t2i_op_attention.
 */
t2i_status t2i_op_cross_attention(int32_t dtype, int32_t heads, int32_t head_dim,
                                  int32_t n_seq, const int32_t* q_start,
                                  const int32_t* q_len, const int32_t* k_start,
                                  const int32_t* k_len, const void* q, int32_t ldq,
                                  const void* k, int32_t ldk, const void* v,
                                  int32_t ldv, void* o, int32_t ldo, void* stream);

/*
 * The DiT block's cross-attention together with its query projection (Sec. 4's
 * model `forward`): q = A W^T + b for the query rows, then the operation of
 * t2i_op_cross_attention with those queries, bf16 only.  The queries are
 * kept multiplied by log2(e)/sqrt(head_dim) (rounded once to bf16, as the
 * model's projection writes them), so the softmax takes base-2 exponentials
 * of the scores directly.
 *   A [M, K] (row stride lda) with M = the largest q_start[s] + q_len[s];
 *   W [heads*head_dim, K] (row stride ldw), bias [heads*head_dim];
 *   K % 64 == 0, lda, ldw >= K and multiples of 8; text of 1 .. 128 keys per
 *   sequence (k_len), key starts % 8 == 0; K/V layouts (V given transposed),
 *   ldk, ldv, ldo and the 2^31-byte limits as for t2i_op_attention.
 * fused = 0: the projection writes the queries to q_buf [M, ldq] (caller-
 *   owned, ldq >= heads*head_dim, % 8 == 0), then the cross-attention kernel
 *   reads them: two launches.
 * fused = 1: one kernel; the queries never leave the chip (q_buf unused, may
 *   be NULL).  Needs head_dim 72, K % 192 == 0, sequences contiguous from
 *   row 0 whose lengths are multiples of 256, 16-byte aligned A, W, K, V and o,
 *   8-byte aligned bias, else T2I_ERR_SHAPE.  Both settings give the
 *   same bits; the model takes the fused one from 2048 rows wherever it
 *   applies.
 */
t2i_status t2i_op_linear_cross_attention(int32_t fused, int32_t heads, int32_t head_dim,
                                         int32_t n_seq, const int32_t* q_start,
                                         const int32_t* q_len, const int32_t* k_start,
                                         const int32_t* k_len, int32_t K, const void* A,
                                         int32_t lda, const void* W, int32_t ldw,
                                         const void* bias, const void* k, int32_t ldk,
                                         const void* v, int32_t ldv, void* q_buf,
                                         int32_t ldq, void* o, int32_t ldo, void* stream);

/*
 * LayerNorm (no affine, biased variance) fused with adaLN modulation:
 * out = (x - mean) / sqrt(var + eps) * (1 + scale) + shift per row of
 * x [rows, D] fp32; shift, scale fp32 [D]; out dtype (bf16 or fp32) [rows, D].
 * D % 4 == 0, D <= 3072; x and shift 16-byte aligned, out 8-byte (bf16) or
 * 16-byte (fp32) aligned.
 */
t2i_status t2i_op_ln_modulate(int32_t dtype, int32_t rows, int32_t D,
                              const float* x, const float* shift,
                              const float* scale, float eps, void* out,
                              void* stream);

/*
 * LoRA weight update merged on the device before sampling (the paper's
 * weight-update adapters, Sec. 2.2 / Sec. 3, which modify base-model weights
 * before inference): W <- W + alpha * B A for one linear layer, in place.
 *   W [n_out, n_in] with row stride ldw, A [rank, n_in] (row stride n_in),
 *   B [n_out, rank] (row stride rank), all of dtype (bf16 or fp32);
 *   1 <= rank <= 128.  The product is accumulated in fp32 over rank, added to
 *   W in fp32 and rounded once to W's dtype (round-to-nearest-even).
 * W is caller-owned memory (e.g. a tensor bound to a t2i_dit handle: merge
 * between calls, not during one).
 */
t2i_status t2i_op_lora_merge(int32_t dtype, int32_t n_out, int32_t n_in, int32_t rank,
                             float alpha, void* W, int32_t ldw, const void* A,
                             const void* B, void* stream);

/*
 * The LoRA merge of t2i_op_lora_merge for n weights of one shape (an adapter
 * applied to every layer of one kind: n_out, n_in, rank, ldw shared), weight
 * i at W[i] with its own A[i], B[i] -- host arrays of n device pointers.
 * Results are those of n t2i_op_lora_merge calls, bitwise; one launch per 64
 * weights instead of one each.  The weights must not overlap.
 */
t2i_status t2i_op_lora_merge_batch(int32_t dtype, int32_t n, int32_t n_out, int32_t n_in,
                                   int32_t rank, float alpha, void* const* W, int32_t ldw,
                                   const void* const* A, const void* const* B, void* stream);

/*
 * Memory-counter calibration (not part of the denoising step): reads `bytes`
 * of src (device, 16-byte aligned; a multiple of 1024 below 2 GiB) exactly
 * once through the direct HBM -> LDS load path that the GEMM and attention
 * kernels use, and writes 1024 floats of no meaning to sink (device).  A
 * profiler's fetched-bytes counter read on this launch gives the factor that
 * turns the counter into bytes for kernels loading this way.
 */
t2i_status t2i_op_dma_read(const void* src, size_t bytes, float* sink, void* stream);

const char* t2i_ops_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* T2I_OPS_H */
