// C ABI of the denoising step: argument validation, workspace layout and the
// launch sequence of one step / one sampling loop on the caller's stream.
// Nothing here computes model values on the host: every number of the path is
// produced by the kernels in gemm.hip, attention.hip and pointwise.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <bitset>
#include <climits>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <utility>
#include <vector>

#include "../../include/t2i_dit.h"
#include "../../include/t2i_ops.h"
#include "t2i_internal.h"

using namespace t2i;

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// ---------------------------------------------------------------------------
// weight table

struct WDesc {
  std::string name;
  int64_t shape[4];
  int nd;
};

std::vector<WDesc> weight_table(const t2i_dit_config& c) {
  std::vector<WDesc> t;
  auto add = [&](const std::string& n, int64_t a, int64_t b = 0) {
    WDesc d;
    d.name = n;
    d.shape[0] = a;
    d.shape[1] = b;
    d.shape[2] = d.shape[3] = 0;
    d.nd = b ? 2 : 1;
    t.push_back(d);
  };
  const int64_t D = c.hidden, F = c.mlp_hidden, P = (int64_t)c.patch * c.patch * c.latent_channels;
  add("x_embed.w", D, P);
  add("x_embed.b", D);
  add("t_embed.w1", D, c.freq_dim);
  add("t_embed.b1", D);
  add("t_embed.w2", D, D);
  add("t_embed.b2", D);
  add("y_embed.w", D, c.text_dim);
  add("y_embed.b", D);
  for (int b = 0; b < c.depth; ++b) {
    const std::string p = "blocks." + std::to_string(b) + ".";
    if (c.arch == T2I_ARCH_CROSS_DIT) {
      add(p + "ada.w", 6 * D, D);
      add(p + "ada.b", 6 * D);
      add(p + "attn.qkv.w", 3 * D, D);
      add(p + "attn.qkv.b", 3 * D);
      add(p + "attn.o.w", D, D);
      add(p + "attn.o.b", D);
      add(p + "xattn.q.w", D, D);
      add(p + "xattn.q.b", D);
      add(p + "xattn.kv.w", 2 * D, D);
      add(p + "xattn.kv.b", 2 * D);
      add(p + "xattn.o.w", D, D);
      add(p + "xattn.o.b", D);
      add(p + "mlp.fc1.w", F, D);
      add(p + "mlp.fc1.b", F);
      add(p + "mlp.fc2.w", D, F);
      add(p + "mlp.fc2.b", D);
    } else {
      for (const char* s : {"txt", "img"}) {
        const std::string q = p + s + ".";
        add(q + "ada.w", 6 * D, D);
        add(q + "ada.b", 6 * D);
        add(q + "qkv.w", 3 * D, D);
        add(q + "qkv.b", 3 * D);
        add(q + "o.w", D, D);
        add(q + "o.b", D);
        add(q + "fc1.w", F, D);
        add(q + "fc1.b", F);
        add(q + "fc2.w", D, F);
        add(q + "fc2.b", D);
      }
    }
  }
  add("final.ada.w", 2 * D, D);
  add("final.ada.b", 2 * D);
  add("final.out.w", P, D);
  add("final.out.b", P);
  return t;
}

// indices into the table
enum { W_PE = 0, B_PE, W_T1, B_T1, W_T2, B_T2, W_Y, B_Y, W_BLOCK0 };
enum { X_ADA = 0, X_ADA_B, X_QKV, X_QKV_B, X_O, X_O_B, X_XQ, X_XQ_B, X_XKV, X_XKV_B, X_XO, X_XO_B,
       X_FC1, X_FC1_B, X_FC2, X_FC2_B, X_PER_BLOCK };
enum { J_ADA = 0, J_ADA_B, J_QKV, J_QKV_B, J_O, J_O_B, J_FC1, J_FC1_B, J_FC2, J_FC2_B, J_PER_STREAM };

int per_block(const t2i_dit_config& c) {
  return c.arch == T2I_ARCH_CROSS_DIT ? X_PER_BLOCK : 2 * J_PER_STREAM;
}
int final_base(const t2i_dit_config& c) { return W_BLOCK0 + c.depth * per_block(c); }
int mod_width(const t2i_dit_config& c) {
  const int per = c.arch == T2I_ARCH_CROSS_DIT ? 6 : 12;
  return c.depth * per * c.hidden + 2 * c.hidden;
}

const char* check_config(const t2i_dit_config* c) {
  if (!c) return "config is NULL";
  if (c->struct_size != sizeof(t2i_dit_config)) return "config struct_size mismatch";
  if (c->arch != T2I_ARCH_CROSS_DIT && c->arch != T2I_ARCH_MMDIT) return "bad arch";
  if (c->dtype != T2I_F32 && c->dtype != T2I_BF16) return "bad dtype";
  if (c->latent_channels < 1 || c->patch < 1) return "bad latent_channels/patch";
  if (c->patch * c->patch * c->latent_channels > 64) return "p*p*C must be <= 64";
  if (c->hidden < 64 || c->hidden % 64 || c->hidden > 3072) return "hidden must be a multiple of 64 in [64, 3072]";
  if (c->heads < 1 || c->heads * c->head_dim != c->hidden) return "heads * head_dim != hidden";
  if (c->head_dim != 32 && c->head_dim != 64 && c->head_dim != 72 && c->head_dim != 128 && c->head_dim != 8)
    return "head_dim must be one of 8, 32, 64, 72, 128";
  if (c->depth < 1 || c->depth > 256) return "bad depth";
  if (c->mlp_hidden < 64 || c->mlp_hidden % 64) return "mlp_hidden must be a positive multiple of 64";
  if (c->text_dim < 64 || c->text_dim % 64) return "text_dim must be a positive multiple of 64";
  if (c->text_tokens < 1 || c->text_tokens > 4096) return "bad text_tokens";
  if (c->freq_dim < 8 || c->freq_dim % 8) return "freq_dim must be a positive multiple of 8";
  if (c->max_tokens < 1) return "bad max_tokens";
  if (c->max_requests < 1 || c->max_requests > T2I_MAX_REQ) return "bad max_requests";
  if (c->max_steps < 1 || c->max_steps > 10000) return "bad max_steps";
  if (!(c->ln_eps > 0.f) || !(c->t_scale > 0.f)) return "bad ln_eps/t_scale";
  if (c->arch == T2I_ARCH_MMDIT && c->dtype != T2I_BF16) return "MMDiT runs in bf16 only";
  if (c->dtype == T2I_BF16 && c->text_tokens % 8) return "bf16 models need text_tokens % 8 == 0";
  if (c->dtype == T2I_BF16) {
    // bf16 attention addresses q|k and V^T with byte offsets below 2^31
    const size_t rows = (size_t)c->max_tokens +
                        (c->arch == T2I_ARCH_MMDIT ? (size_t)2 * c->max_requests * c->text_tokens : 0);
    if ((size_t)4 * (rows + 64) * c->hidden > 0x7fffffff ||
        (size_t)2 * c->hidden * ((rows + 63) / 64 * 64) > 0x7fffffff)
      return "max_tokens too large for the bf16 attention's 2 GiB operand limit";
  }
  return nullptr;
}

// ---------------------------------------------------------------------------
// workspace layout

struct Layout {
  size_t x, x0, xf, h, xb, qkv, vt, o, u, ytxt, kv, vtt, rope, pe, splitk, tfreq, th1, tsc, mod,
      partial, total;
  size_t splitk_floats = 0;
  bool has_xf = false;          // xf allocated (cross-DiT, several requests)
  int ldvt = 0, ldvt_txt = 0;   // token strides of the transposed V buffers
};

Layout layout(const t2i_dit_config& c) {
  Layout L{};
  const size_t A = c.dtype == T2I_BF16 ? 2 : 4;
  const size_t D = c.hidden, F = c.mlp_hidden;
  const bool mm = c.arch == T2I_ARCH_MMDIT;
  // cross-DiT: the prompts plus one shared unconditional prompt; MMDiT: a
  // text stream per request and guidance branch
  const size_t txt_rows = (size_t)(mm ? 2 * c.max_requests : c.max_requests + 1) * c.text_tokens;
  size_t rows = c.max_tokens;
  if (mm) rows += txt_rows;   // residual rows: text stream, then image stream
  const size_t Tt = (size_t)c.max_steps * c.max_requests;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  L.x = take(rows * D * 4);
  L.x0 = take(rows * D * 4);
  // cross-DiT batches of several requests: the image rows of every request
  // in the call's layout while the blocks run on the computing requests only
  // (compacted; see step_body)
  L.has_xf = !mm && c.max_requests > 1;
  L.xf = take(L.has_xf ? (size_t)c.max_tokens * D * 4 : 0);
  L.h = take(rows * D * A);
  L.xb = take(c.dtype == T2I_BF16 ? rows * D * 2 : 0);
  L.qkv = take(rows * 3 * D * A);
  // bf16 attention reads V transposed: [D][ldvt], token index contiguous
  L.ldvt = (int)((rows + 63) / 64 * 64);
  L.ldvt_txt = (int)((txt_rows + 63) / 64 * 64);
  const bool bfv = c.dtype == T2I_BF16;
  L.vt = take(bfv ? D * (size_t)L.ldvt * 2 : 0);
  L.o = take(rows * D * A);
  L.u = take(rows * F * A);
  L.ytxt = take(txt_rows * D * (mm ? 4 : A));   // MMDiT keeps the projected text in fp32
  L.kv = take(c.arch == T2I_ARCH_CROSS_DIT ? (size_t)c.depth * txt_rows * 2 * D * A : 0);
  L.vtt = take(c.arch == T2I_ARCH_CROSS_DIT && bfv ? (size_t)c.depth * D * L.ldvt_txt * 2 : 0);
  L.rope = take(mm ? (size_t)(4096 / c.patch) * (c.head_dim / 4) * sizeof(float2) : 0);
  L.pe = take(mm ? 0 : (size_t)(4096 / c.patch) * (c.hidden / 4) * sizeof(float2));
  // split-K partial sums of the text projections against long K (the MMDiT
  // text stream's narrow layers; the cross-DiT's caption projection, K =
  // text_dim): at most 4 slices of up to 2047 rows
  L.splitk_floats = (mm || bfv) ? (size_t)4 * std::min<size_t>(txt_rows, 2047) * D : 0;
  L.splitk = take(L.splitk_floats * 4);
  L.tfreq = take(Tt * c.freq_dim * 4);
  L.th1 = take(Tt * D * 4);
  L.tsc = take(Tt * D * 4);
  L.mod = take(Tt * mod_width(c) * 4);
  L.partial = take(((size_t)c.max_tokens / kCacheRowsPerBlock + c.max_requests + 1) * 2 * 8);
  L.total = off;
  return L;
}

}  // namespace

// ---------------------------------------------------------------------------

struct t2i_dit {
  t2i_dit_config cfg;
  std::vector<const void*> w;
  char* ws = nullptr;
  size_t ws_bytes = 0;
  Layout L{};
  std::string err;
  std::vector<CacheHeader> hdr_host;
  // kernel timing
  uint32_t prof_mask = 0;
  std::vector<hipEvent_t> ev_pool;               // created on demand, reused
  size_t ev_used = 0;
  std::vector<std::pair<int, size_t>> ev_pairs;  // (class, index of start event)
  // layer residency: per block resident / loading / evicted, the event after
  // each block's queued copy, and the host tier the copies read
  enum : uint8_t { BLK_RESIDENT = 0, BLK_LOADING = 1, BLK_EVICTED = 2 };
  std::vector<uint8_t> blk;
  std::vector<hipEvent_t> blk_ev;
  const char* host_blocks = nullptr;
  char* arena = nullptr;
  size_t blk_bytes = 0;
  std::vector<size_t> blk_off;   // packed offset of each tensor of a block

  ~t2i_dit() {
    for (size_t b = 0; b < blk_ev.size(); ++b)
      if (blk_ev[b]) {
        if (blk[b] == BLK_LOADING) (void)hipEventSynchronize(blk_ev[b]);
        (void)hipEventDestroy(blk_ev[b]);
      }
    for (hipEvent_t e : ev_pool) (void)hipEventDestroy(e);
  }

  template <typename T>
  T* at(size_t off) const { return (T*)(ws + off); }
  bool bf() const { return cfg.dtype == T2I_BF16; }
  size_t act() const { return bf() ? 2 : 4; }
};

namespace {

thread_local std::string g_ops_err;

t2i_status fail(t2i_dit* h, t2i_status s, const std::string& msg) {
  if (h) h->err = msg;
  return s;
}

#define HIP_TRY(h, expr)                                                              \
  do {                                                                                \
    hipError_t e_ = (expr);                                                           \
    if (e_ != hipSuccess)                                                             \
      return fail((h), T2I_ERR_DEVICE, std::string(#expr ": ") + hipGetErrorString(e_)); \
  } while (0)

// One call's request geometry.
struct Plan {
  int n_req = 0, branches = 1, T_img = 0, rows = 0, txt_rows = 0;
  float guidance = 1.f;
  ReqMap rm{};
  SeqMap img{};      // image rows (branch-major) -> sequence -> modulation row
  SeqMap txt{};      // MMDiT text-stream rows (branch-major), same sequences
  AttnMap self{}, cross{};
  AttnMap joint{};   // MMDiT: per sequence a text and an image query group,
                     // keys = the sequence's text rows, then its image rows
  int grid_max = 0;  // largest grid side (length of the position tables)
  const t2i_control* ctl = nullptr;   // validated callback input, or NULL
  size_t lat_floats = 0;
  // blocks >= defer_from are still loading: their modulation rows (cond_rows
  // of them) and text K/V are computed right before the block, after its load
  // event; `done` marks the deferred blocks already prepared in this call
  int defer_from = INT_MAX;
  int cond_rows = 0;
  mutable std::bitset<256> done;
};

t2i_status build_plan(t2i_dit* h, int n_req, const int32_t* lat_h, const int32_t* lat_w,
                      float guidance, Plan& P) {
  const t2i_dit_config& c = h->cfg;
  if (n_req < 1 || n_req > c.max_requests) return fail(h, T2I_ERR_SHAPE, "n_req out of range");
  if (!lat_h || !lat_w) return fail(h, T2I_ERR_INVALID_ARG, "lat_h/lat_w is NULL");
  if (!std::isfinite(guidance)) return fail(h, T2I_ERR_INVALID_ARG, "guidance not finite");
  P.n_req = n_req;
  P.guidance = guidance;
  P.branches = guidance == 1.f ? 1 : 2;
  if (n_req * P.branches > kMaxSeq) return fail(h, T2I_ERR_SHAPE, "too many sequences");
  int tok = 0;
  size_t lat = 0;
  P.rm.n = n_req;
  for (int r = 0; r < n_req; ++r) {
    if (lat_h[r] < c.patch || lat_w[r] < c.patch || lat_h[r] % c.patch || lat_w[r] % c.patch)
      return fail(h, T2I_ERR_SHAPE, "latent size must be a positive multiple of patch");
    if (lat_h[r] > 4096 || lat_w[r] > 4096) return fail(h, T2I_ERR_SHAPE, "latent too large");
    const int n = (lat_h[r] / c.patch) * (lat_w[r] / c.patch);
    if (h->bf() && n % 8)
      return fail(h, T2I_ERR_SHAPE, "bf16 models need image tokens per request % 8 == 0");
    P.rm.tok_off[r] = tok;
    P.rm.lat_off[r] = (int)lat;
    P.rm.h[r] = lat_h[r];
    P.rm.w[r] = lat_w[r];
    P.rm.modrow[r] = r;
    P.rm.dt[r] = 0.f;
    tok += n;
    lat += (size_t)c.latent_channels * lat_h[r] * lat_w[r];
  }
  P.rm.tok_off[n_req] = tok;
  P.rm.tokens_total = tok;
  P.rm.branches = P.branches;
  P.T_img = tok;
  P.rows = tok * P.branches;
  P.lat_floats = lat;
  if (P.rows > c.max_tokens) return fail(h, T2I_ERR_SHAPE, "image tokens exceed max_tokens");
  const int M = c.text_tokens;
  P.txt_rows = n_req * M + (P.branches == 2 ? M : 0);
  P.img.n = n_req * P.branches;
  P.self.n = P.cross.n = P.img.n;
  for (int br = 0; br < P.branches; ++br)
    for (int r = 0; r < n_req; ++r) {
      const int s = br * n_req + r;
      const int start = br * tok + P.rm.tok_off[r];
      const int len = P.rm.tok_off[r + 1] - P.rm.tok_off[r];
      P.img.start[s] = start;
      P.img.modrow[s] = r;
      P.self.q_start[s] = P.cross.q_start[s] = start;
      P.self.q_len[s] = P.cross.q_len[s] = len;
      P.self.k_start[s] = start;
      P.self.k_len[s] = len;
      P.cross.k_start[s] = br == 0 ? r * M : n_req * M;
      P.cross.k_len[s] = M;
    }
  P.img.start[P.img.n] = P.rows;
  attention_tiles(P.self, h->bf(), c.heads, 0);
  attention_tiles(P.cross, h->bf(), c.heads, 1);
  if (c.arch == T2I_ARCH_MMDIT) {
    // residual rows are stream-major: text rows [0, txt_rows) with sequence s
    // at s*M, then the image rows (offset txt_rows) in the cross-DiT order
    if (2 * P.img.n > kMaxSeq) return fail(h, T2I_ERR_SHAPE, "too many sequences for MMDiT");
    P.txt_rows = P.img.n * M;
    P.txt.n = P.img.n;
    for (int s = 0; s < P.img.n; ++s) {
      P.txt.start[s] = s * M;
      P.txt.modrow[s] = s % n_req;
      const int ist = P.txt_rows + P.img.start[s], ilen = P.img.start[s + 1] - P.img.start[s];
      for (int g = 0; g < 2; ++g) {
        const int q = 2 * s + g;
        P.joint.q_start[q] = g ? ist : s * M;
        P.joint.q_len[q] = g ? ilen : M;
        P.joint.k_start[q] = s * M;
        P.joint.k_len[q] = M;
        P.joint.k2_start[q] = ist;
        P.joint.k2_len[q] = ilen;
      }
    }
    P.txt.start[P.txt.n] = P.txt_rows;
    P.joint.n = 2 * P.img.n;
    attention_tiles(P.joint, true, c.heads, 0);
  }
  for (int r = 0; r < n_req; ++r)
    P.grid_max = std::max(P.grid_max, std::max(lat_h[r], lat_w[r]) / c.patch);
  return T2I_OK;
}

void set_modrows(Plan& P, int base) {
  for (int r = 0; r < P.n_req; ++r) P.rm.modrow[r] = base + r;
  for (int s = 0; s < P.img.n; ++s) P.img.modrow[s] = base + (s % P.n_req);
  for (int s = 0; s < P.txt.n; ++s) P.txt.modrow[s] = base + (s % P.n_req);
}

bool is_mmdit(const t2i_dit* h) { return h->cfg.arch == T2I_ARCH_MMDIT; }

// Patch embedding of the call's latents into x0 (and `copies` copies into xi);
// the cross-attention DiT adds its 2D sin-cos position embedding.
hipError_t embed(t2i_dit* h, const Plan& P, const float* lat, float* x0, float* xi, int copies,
                 hipStream_t st) {
  const t2i_dit_config& c = h->cfg;
  float2* pe = is_mmdit(h) ? nullptr : h->at<float2>(h->L.pe);
  return launch_embed(lat, P.rm, h->w[W_PE], h->w[B_PE], h->bf(), c.hidden, c.latent_channels,
                      c.patch, pe, P.grid_max, x0, xi, copies, st);
}
// first residual row of the image stream
int img_row0(const t2i_dit* h, const Plan& P) { return is_mmdit(h) ? P.txt_rows : 0; }

// Callback input after block b: wait for its producer's event (if any) at this
// point only, then add the residual to the image stream.
hipError_t inject_control(t2i_dit* h, const Plan& P, int b, hipStream_t st) {
  const t2i_control* c = P.ctl;
  if (!c) return hipSuccess;
  for (int i = 0; i < c->n; ++i) {
    if (c->blocks[i] != b) continue;
    if (c->ready && c->ready[i]) {
      hipError_t e = hipStreamWaitEvent(st, (hipEvent_t)c->ready[i], 0);
      if (e != hipSuccess) return e;
    }
    float* xi = h->at<float>(h->L.x) + (size_t)img_row0(h, P) * h->cfg.hidden;
    return launch_add_inplace(xi, c->residuals[i], (size_t)P.rows * h->cfg.hidden, st);
  }
  return hipSuccess;
}

Epi make_epi() {
  Epi e;
  std::memset(&e, 0, sizeof(e));
  return e;
}

// The fused query projection + cross-attention's view of a cross-attention
// map (text K row-major with stride ldk, V^T with stride ldvt, output o);
// a map with second key segments gets n = 0, which the launcher rejects.
XAttnArgs make_xattn(const AttnMap& m, const void* k, int ldk, const void* vt, int ldvt, void* o,
                     int ldo) {
  XAttnArgs a;
  std::memset(&a, 0, sizeof(a));
  a.K = (const bf16*)k;
  a.ldk = ldk;
  a.Vt = (const bf16*)vt;
  a.ldvt = ldvt;
  a.O = (bf16*)o;
  a.ldo = ldo;
  a.n = m.n;
  for (int s = 0; s < m.n; ++s) {
    a.q_start[s] = m.q_start[s];
    a.q_len[s] = m.q_len[s];
    a.k_start[s] = m.k_start[s];
    a.k_len[s] = m.k_len[s];
    if (m.k2_len[s]) a.n = 0;
  }
  return a;
}

// y = A W^T + b with the config's operand type.  allow_split lets a
// short-M, long-K layer split K (MMDiT text stream).
hipError_t linear(t2i_dit* h, const void* A, int lda, int wi, int M, int N, int K, int kind,
                  Epi epi, hipStream_t st, bool allow_split = false) {
  const void* W = h->w[wi];
  const void* B = h->w[wi + 1];
  if (h->bf())
    return launch_gemm_bf16((const bf16*)A, lda, (const bf16*)W, K, (const bf16*)B, M, N, K, kind,
                            epi, allow_split ? h->at<float>(h->L.splitk) : nullptr,
                            allow_split ? h->L.splitk_floats : 0, st);
  return launch_gemm_f32((const float*)A, lda, W, K, false, B, M, N, K, kind, epi, st);
}

// Block b's adaLN chunks of `rows` conditioning rows (silu(c) in tsc) into
// the modulation table.
hipError_t block_modulation(t2i_dit* h, int b, int rows, hipStream_t st) {
  const t2i_dit_config& c = h->cfg;
  const int D = c.hidden, pb = per_block(c);
  const float* tsc = h->at<float>(h->L.tsc);
  float* mod = h->at<float>(h->L.mod);
  Epi e = make_epi();
  e.ldo = mod_width(c);
  if (c.arch == T2I_ARCH_CROSS_DIT) {
    e.out = mod + (size_t)b * 6 * D;
    const int wi = W_BLOCK0 + b * pb + X_ADA;
    return launch_linear_rows(tsc, D, h->w[wi], D, h->bf(), h->w[wi + 1], rows, 6 * D, D,
                              EPI_STORE, e, st);
  }
  for (int s = 0; s < 2; ++s) {
    e.out = mod + (size_t)b * 12 * D + (size_t)s * 6 * D;
    const int wi = W_BLOCK0 + b * pb + s * J_PER_STREAM + J_ADA;
    hipError_t err = launch_linear_rows(tsc, D, h->w[wi], D, h->bf(), h->w[wi + 1], rows, 6 * D,
                                        D, EPI_STORE, e, st);
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

// The adaLN chunks of blocks [b0, b1) in grouped launches (one group per
// block, per stream for MMDiT); bitwise the per-block block_modulation.
hipError_t blocks_modulation(t2i_dit* h, int b0, int b1, int rows, hipStream_t st) {
  const t2i_dit_config& c = h->cfg;
  const int D = c.hidden, pb = per_block(c);
  const bool mm = c.arch != T2I_ARCH_CROSS_DIT;
  const float* tsc = h->at<float>(h->L.tsc);
  float* mod = h->at<float>(h->L.mod);
  Epi e = make_epi();
  e.ldo = mod_width(c);
  PtrGroup g;
  int n = 0;
  auto flush = [&]() {
    hipError_t err = launch_linear_rows_group(tsc, D, g, n, D, h->bf(), rows, 6 * D, D, e, st);
    n = 0;
    return err;
  };
  for (int b = b0; b < b1; ++b)
    for (int s = 0; s < (mm ? 2 : 1); ++s) {
      const int wi = mm ? W_BLOCK0 + b * pb + s * J_PER_STREAM + J_ADA : W_BLOCK0 + b * pb + X_ADA;
      g.W[n] = h->w[wi];
      g.bias[n] = h->w[wi + 1];
      g.out[n] = mod + (size_t)b * (mm ? 12 : 6) * D + (size_t)s * 6 * D;
      g.vt[n] = nullptr;
      if (++n == kMaxGroups) {
        hipError_t err = flush();
        if (err != hipSuccess) return err;
      }
    }
  return flush();
}

// The call's stream waits for block b's queued load, if any.
hipError_t wait_block(t2i_dit* h, int b, hipStream_t st) {
  if (h->blk[b] != t2i_dit::BLK_LOADING) return hipSuccess;
  return hipStreamWaitEvent(st, h->blk_ev[b], 0);
}

// Conditioning of `rows` timesteps (rows <= max_steps * max_requests):
// silu(c) into tsc and the adaLN chunks of blocks [0, min(n_blocks_mod,
// defer_from)) into the modulation table.
t2i_status conditioning(t2i_dit* h, const double* t_host, int rows, int n_blocks_mod,
                        int defer_from, hipStream_t st) {
  const t2i_dit_config& c = h->cfg;
  const int D = c.hidden, fd = c.freq_dim;
  float* tfreq = h->at<float>(h->L.tfreq);
  float* th1 = h->at<float>(h->L.th1);
  float* tsc = h->at<float>(h->L.tsc);
  float* mod = h->at<float>(h->L.mod);
  const bool wb = h->bf();
  HIP_TRY(h, launch_timestep_freq(t_host, rows, fd, (double)c.t_scale, tfreq, st));
  Epi e = make_epi();
  e.out = th1;
  e.ldo = D;
  HIP_TRY(h, launch_linear_rows(tfreq, fd, h->w[W_T1], fd, wb, h->w[B_T1], rows, D, fd, EPI_SILU, e, st));
  e.out = tsc;
  HIP_TRY(h, launch_linear_rows(th1, D, h->w[W_T2], D, wb, h->w[B_T2], rows, D, D, EPI_SILU, e, st));
  const int mw = mod_width(c);
  e.ldo = mw;
  const int nbm = std::min(n_blocks_mod, defer_from);
  for (int b = 0; b < nbm; ++b) HIP_TRY(h, wait_block(h, b, st));
  HIP_TRY(h, blocks_modulation(h, 0, nbm, rows, st));
  e.out = mod + (size_t)(mw - 2 * D);
  const int fb = final_base(c);
  HIP_TRY(h, launch_linear_rows(tsc, D, h->w[fb], D, wb, h->w[fb + 1], rows, 2 * D, D, EPI_STORE, e, st));
  return T2I_OK;
}

// Cross-DiT block b's text K/V from the projected text in ytxt.
hipError_t block_text_kv(t2i_dit* h, const Plan& P, int b, hipStream_t st) {
  const t2i_dit_config& c = h->cfg;
  const int D = c.hidden;
  const size_t txt_rows_max = (size_t)(c.max_requests + 1) * c.text_tokens;
  Epi e = make_epi();
  e.out = h->at<char>(h->L.kv) + (size_t)b * txt_rows_max * 2 * D * h->act();
  e.ldo = 2 * D;
  int kind = EPI_STORE;
  if (h->bf()) {   // k row-major [rows, D], v transposed [D][ldvt_txt]
    kind = EPI_SPLIT_VT;
    e.ldo = D;
    e.vt = h->at<bf16>(h->L.vtt) + (size_t)b * D * h->L.ldvt_txt;
    e.ldvt = h->L.ldvt_txt;
    e.vcol0 = D;
  }
  return linear(h, h->at<char>(h->L.ytxt), D, W_BLOCK0 + b * X_PER_BLOCK + X_XKV, P.txt_rows,
                2 * D, D, kind, e, st);
}

// Text projection and (cross-DiT) the text K/V of blocks [0, min(nb,
// P.defer_from)).
t2i_status text_prep(t2i_dit* h, const Plan& P, const void* prompt, int nb, hipStream_t st) {
  const t2i_dit_config& c = h->cfg;
  const int D = c.hidden, M = c.text_tokens;
  char* ytxt = h->at<char>(h->L.ytxt);
  Epi e = make_epi();
  e.out = ytxt;
  e.ldo = D;
  if (is_mmdit(h)) {
    // fp32 initial text stream of every sequence (unconditional: the bias),
    // copied into the residual at the start of each step; RoPE table
    HIP_TRY(h, linear(h, prompt, c.text_dim, W_Y, P.n_req * M, D, c.text_dim, EPI_STORE_F32, e,
                      st));
    if (P.branches == 2)
      HIP_TRY(h, launch_bias_rows_f32(h->w[B_Y], h->bf(), P.n_req * M, D,
                                      (float*)ytxt + (size_t)P.n_req * M * D, st));
    HIP_TRY(h, launch_rope_table(h->at<float2>(h->L.rope), P.grid_max, c.head_dim / 4, st));
    return T2I_OK;
  }
  // a few hundred rows against K = text_dim: K split over workgroups
  HIP_TRY(h, linear(h, prompt, c.text_dim, W_Y, P.n_req * M, D, c.text_dim, EPI_STORE, e, st,
                    /*allow_split=*/true));
  if (P.branches == 2)
    HIP_TRY(h, launch_broadcast_rows(h->w[B_Y], h->bf(), M, D,
                                     ytxt + (size_t)P.n_req * M * D * h->act(), st));
  if (c.arch != T2I_ARCH_CROSS_DIT) return T2I_OK;
  const int nkv = std::min(nb, P.defer_from);
  if (!h->bf() || !gemm_bf16_groupable(P.txt_rows, 2 * D, EPI_SPLIT_VT)) {
    for (int b = 0; b < nkv; ++b) HIP_TRY(h, block_text_kv(h, P, b, st));
    return T2I_OK;
  }
  // every block's K / V from one grouped launch (per 64 blocks)
  const size_t txt_rows_max = (size_t)(c.max_requests + 1) * M;
  Epi g_epi = make_epi();
  g_epi.ldo = D;
  g_epi.ldvt = h->L.ldvt_txt;
  g_epi.vcol0 = D;
  PtrGroup g;
  for (int b0 = 0; b0 < nkv; b0 += kMaxGroups) {
    const int n = std::min(kMaxGroups, nkv - b0);
    for (int i = 0; i < n; ++i) {
      const int b = b0 + i, wi = W_BLOCK0 + b * X_PER_BLOCK + X_XKV;
      g.W[i] = h->w[wi];
      g.bias[i] = h->w[wi + 1];
      g.out[i] = h->at<char>(h->L.kv) + (size_t)b * txt_rows_max * 2 * D * h->act();
      g.vt[i] = h->at<bf16>(h->L.vtt) + (size_t)b * D * h->L.ldvt_txt;
    }
    HIP_TRY(h, launch_gemm_bf16_group(h->at<bf16>(h->L.ytxt), D, g, n, D, P.txt_rows, 2 * D, D,
                                      EPI_SPLIT_VT, g_epi, st));
  }
  return T2I_OK;
}

// Before the first use of block b's weights in a call: when the block is
// still loading, wait for its copy and compute its deferred modulation rows
// and text K/V.
t2i_status ensure_block(t2i_dit* h, const Plan& P, int b, hipStream_t st) {
  if (b < P.defer_from || P.done[b]) return T2I_OK;
  HIP_TRY(h, wait_block(h, b, st));
  HIP_TRY(h, block_modulation(h, b, P.cond_rows, st));
  if (h->cfg.arch == T2I_ARCH_CROSS_DIT) HIP_TRY(h, block_text_kv(h, P, b, st));
  P.done[b] = true;
  return T2I_OK;
}

// Event pair around one launch of a timed kernel class.
hipError_t prof_mark(t2i_dit* h, int cls, bool start, hipStream_t st) {
  if (!(h->prof_mask & (1u << cls))) return hipSuccess;
  if (h->ev_used == h->ev_pool.size()) {
    hipEvent_t e;
    hipError_t err = hipEventCreate(&e);
    if (err != hipSuccess) return err;
    h->ev_pool.push_back(e);
  }
  const size_t i = h->ev_used++;
  if (start) h->ev_pairs.push_back({cls, i});
  return hipEventRecord(h->ev_pool[i], st);
}

#define TIMED(h, cls, st, expr)                      \
  do {                                               \
    HIP_TRY(h, prof_mark(h, cls, true, st));         \
    HIP_TRY(h, expr);                                \
    HIP_TRY(h, prof_mark(h, cls, false, st));        \
  } while (0)

// Cross-DiT blocks [0, nb) over all image rows of the plan.
t2i_status run_blocks_cross(t2i_dit* h, const Plan& P, int nb, hipStream_t st) {
  const t2i_dit_config& c = h->cfg;
  const int D = c.hidden, F = c.mlp_hidden, R = P.rows, mw = mod_width(c);
  const bool bf = h->bf();
  float* x = h->at<float>(h->L.x);
  char* hb = h->at<char>(h->L.h);
  char* qkv = h->at<char>(h->L.qkv);
  char* o = h->at<char>(h->L.o);
  char* u = h->at<char>(h->L.u);
  bf16* xb = bf ? h->at<bf16>(h->L.xb) : nullptr;
  bf16* vt = bf ? h->at<bf16>(h->L.vt) : nullptr;
  const float* mod = h->at<float>(h->L.mod);
  const size_t A = h->act();
  const size_t txt_rows_max = (size_t)(c.max_requests + 1) * c.text_tokens;
  for (int b = 0; b < nb; ++b) {
    if (t2i_status s = ensure_block(h, P, b, st)) return s;
    const int wb = W_BLOCK0 + b * X_PER_BLOCK;
    const int mo = b * 6 * D;
    // self-attention
    TIMED(h, T2I_K_LN, st, launch_ln_modulate(bf, R, D, x, D, mod, mw, mo + 0 * D, mo + 1 * D,
                                               P.img, hb, D, c.ln_eps, st));
    Epi e = make_epi();
    e.out = qkv;
    if (bf) {   // q (scaled for the softmax) | k row-major [R, 2D], v transposed [D][ldvt]
      e.ldo = 2 * D;
      e.vt = vt;
      e.ldvt = h->L.ldvt;
      e.vcol0 = 2 * D;
      e.qscale = attn_q_scale(c.head_dim);
      e.qcols = D;
      TIMED(h, T2I_K_GEMM_QKV, st, linear(h, hb, D, wb + X_QKV, R, 3 * D, D, EPI_SPLIT_VT, e, st));
      TIMED(h, T2I_K_ATTN_SELF, st,
            launch_attention(bf, 0, c.heads, c.head_dim, P.self, qkv, 2 * D, qkv + D * A, 2 * D, vt,
                             h->L.ldvt, o, D, st, true));
    } else {
      e.ldo = 3 * D;
      TIMED(h, T2I_K_GEMM_QKV, st, linear(h, hb, D, wb + X_QKV, R, 3 * D, D, EPI_STORE, e, st));
      TIMED(h, T2I_K_ATTN_SELF, st,
            launch_attention(bf, 0, c.heads, c.head_dim, P.self, qkv, 3 * D, qkv + D * A, 3 * D,
                             qkv + 2 * D * A, 3 * D, o, D, st, false));
    }
    e = make_epi();
    e.x = x;
    e.ldx = D;
    e.xb = xb;
    e.gate = mod + mo + 2 * D;
    e.ld_gate = mw;
    e.map = P.img;
    TIMED(h, T2I_K_GEMM_O, st, linear(h, o, D, wb + X_O, R, D, D, EPI_RESID_GATED, e, st));
    // cross-attention (query from the raw residual, ungated)
    e = make_epi();
    e.out = qkv;
    e.ldo = D;
    if (bf) {   // the cross-attention query, scaled for the softmax
      e.qscale = attn_q_scale(c.head_dim);
      e.qcols = D;
    }
    const char* kv = h->at<char>(h->L.kv) + (size_t)b * txt_rows_max * 2 * D * A;
    if (bf) {
      // one kernel for the query projection and the cross-attention where
      // the shapes fit it (same bits as the two launches below) and the
      // projection would run on 256-row tiles anyway (from 2048 rows; below,
      // the narrower tiles of the separate projection keep more CUs busy:
      // the 512-px model's 1024 rows make 32 fused workgroups)
      const bf16* vtt = h->at<bf16>(h->L.vtt) + (size_t)b * D * h->L.ldvt_txt;
      const XAttnArgs xa = make_xattn(P.cross, kv, D, vtt, h->L.ldvt_txt, o, D);
      const bf16* wq = (const bf16*)h->w[wb + X_XQ];
      const bf16* bq = (const bf16*)h->w[wb + X_XQ + 1];
      if (R >= 2048 &&
          launch_gemm_xattn(xb, D, wq, D, bq, R, D, D, e, c.heads, c.head_dim, xa, st, true) ==
              hipSuccess) {
        TIMED(h, T2I_K_GEMM_XQ, st,
              launch_gemm_xattn(xb, D, wq, D, bq, R, D, D, e, c.heads, c.head_dim, xa, st));
      } else {
        TIMED(h, T2I_K_GEMM_XQ, st, linear(h, xb, D, wb + X_XQ, R, D, D, EPI_STORE, e, st));
        TIMED(h, T2I_K_ATTN_CROSS, st,
              launch_attention(bf, 1, c.heads, c.head_dim, P.cross, qkv, D, kv, D, vtt,
                               h->L.ldvt_txt, o, D, st, true));
      }
    } else {
      TIMED(h, T2I_K_GEMM_XQ, st, linear(h, x, D, wb + X_XQ, R, D, D, EPI_STORE, e, st));
      TIMED(h, T2I_K_ATTN_CROSS, st,
            launch_attention(bf, 1, c.heads, c.head_dim, P.cross, qkv, D, kv, 2 * D, kv + D * A,
                             2 * D, o, D, st, false));
    }
    e = make_epi();
    e.x = x;
    e.ldx = D;
    TIMED(h, T2I_K_GEMM_XO, st, linear(h, o, D, wb + X_XO, R, D, D, EPI_RESID, e, st));
    // MLP
    TIMED(h, T2I_K_LN, st, launch_ln_modulate(bf, R, D, x, D, mod, mw, mo + 3 * D, mo + 4 * D,
                                               P.img, hb, D, c.ln_eps, st));
    e = make_epi();
    e.out = u;
    e.ldo = F;
    TIMED(h, T2I_K_GEMM_FC1, st, linear(h, hb, D, wb + X_FC1, R, F, D, EPI_GELU, e, st));
    e = make_epi();
    e.x = x;
    e.ldx = D;
    e.gate = mod + mo + 5 * D;
    e.ld_gate = mw;
    e.map = P.img;
    TIMED(h, T2I_K_GEMM_FC2, st, linear(h, u, F, wb + X_FC2, R, D, F, EPI_RESID_GATED, e, st));
    HIP_TRY(h, inject_control(h, P, b, st));
  }
  return T2I_OK;
}

// MMDiT joint blocks [0, nb): per stream (text rows, then image rows of the
// residual) LN-modulate and projections with that stream's weights and
// modulation; RoPE on the image q, k; one joint attention over both.
t2i_status run_blocks_mmdit(t2i_dit* h, const Plan& P, int nb, hipStream_t st) {
  const t2i_dit_config& c = h->cfg;
  const int D = c.hidden, F = c.mlp_hidden, mw = mod_width(c);
  float* x = h->at<float>(h->L.x);
  bf16* hb = h->at<bf16>(h->L.h);
  bf16* qkv = h->at<bf16>(h->L.qkv);
  bf16* o = h->at<bf16>(h->L.o);
  bf16* u = h->at<bf16>(h->L.u);
  bf16* vt = h->at<bf16>(h->L.vt);
  const float* mod = h->at<float>(h->L.mod);
  const float2* rope = h->at<float2>(h->L.rope);
  const int r0s[2] = {0, P.txt_rows}, ns[2] = {P.txt_rows, P.rows};
  const SeqMap* maps[2] = {&P.txt, &P.img};
  for (int b = 0; b < nb; ++b) {
    if (t2i_status s = ensure_block(h, P, b, st)) return s;
    for (int s = 0; s < 2; ++s) {
      const int r0 = r0s[s], R = ns[s], wi = W_BLOCK0 + b * 2 * J_PER_STREAM + s * J_PER_STREAM;
      const int mo = b * 12 * D + s * 6 * D;
      TIMED(h, T2I_K_LN, st, launch_ln_modulate(true, R, D, x + (size_t)r0 * D, D, mod, mw, mo,
                                                 mo + D, *maps[s], hb + (size_t)r0 * D, D,
                                                 c.ln_eps, st));
      Epi e = make_epi();   // q (scaled) | k row-major [rows, 2D], v transposed [D][ldvt]
      e.out = qkv + (size_t)r0 * 2 * D;
      e.ldo = 2 * D;
      e.vt = vt + r0;
      e.ldvt = h->L.ldvt;
      e.vcol0 = 2 * D;
      e.qscale = attn_q_scale(c.head_dim);
      e.qcols = D;
      TIMED(h, T2I_K_GEMM_QKV, st,
            linear(h, hb + (size_t)r0 * D, D, wi + J_QKV, R, 3 * D, D, EPI_SPLIT_VT, e, st));
    }
    HIP_TRY(h, launch_rope_apply(qkv, 2 * D, P.txt_rows, P.rm, c.heads, c.head_dim, c.patch, rope,
                                 st));
    TIMED(h, T2I_K_ATTN_SELF, st,
          launch_attention(true, 0, c.heads, c.head_dim, P.joint, qkv, 2 * D, qkv + D, 2 * D, vt,
                           h->L.ldvt, o, D, st, true));
    for (int s = 0; s < 2; ++s) {
      const int r0 = r0s[s], R = ns[s], wi = W_BLOCK0 + b * 2 * J_PER_STREAM + s * J_PER_STREAM;
      const int mo = b * 12 * D + s * 6 * D;
      Epi e = make_epi();
      e.x = x + (size_t)r0 * D;
      e.ldx = D;
      e.gate = mod + mo + 2 * D;
      e.ld_gate = mw;
      e.map = *maps[s];
      TIMED(h, T2I_K_GEMM_O, st,
            linear(h, o + (size_t)r0 * D, D, wi + J_O, R, D, D, EPI_RESID_GATED, e, st, s == 0));
      TIMED(h, T2I_K_LN, st, launch_ln_modulate(true, R, D, x + (size_t)r0 * D, D, mod, mw,
                                                 mo + 3 * D, mo + 4 * D, *maps[s],
                                                 hb + (size_t)r0 * D, D, c.ln_eps, st));
      Epi f = make_epi();
      f.out = u + (size_t)r0 * F;
      f.ldo = F;
      TIMED(h, T2I_K_GEMM_FC1, st,
            linear(h, hb + (size_t)r0 * D, D, wi + J_FC1, R, F, D, EPI_GELU, f, st));
      e.gate = mod + mo + 5 * D;
      TIMED(h, T2I_K_GEMM_FC2, st,
            linear(h, u + (size_t)r0 * F, F, wi + J_FC2, R, D, F, EPI_RESID_GATED, e, st, s == 0));
    }
    HIP_TRY(h, inject_control(h, P, b, st));
  }
  return T2I_OK;
}

t2i_status run_blocks(t2i_dit* h, const Plan& P, int nb, hipStream_t st) {
  if (h->cfg.arch == T2I_ARCH_CROSS_DIT) return run_blocks_cross(h, P, nb, st);
  return run_blocks_mmdit(h, P, nb, st);
}

size_t cache_bytes(const t2i_dit_config& c, int n_req, int tokens, int branches) {
  return align_up((size_t)n_req * sizeof(CacheHeader)) + align_up((size_t)tokens * c.hidden * 4) +
         (size_t)branches * tokens * c.hidden * 4;
}

struct CachePtrs {
  CacheHeader* hdr;
  float* m_prev;
  float* R;
};

CachePtrs cache_ptrs(const t2i_dit_config& c, void* base, int n_req, int tokens) {
  CachePtrs p;
  char* b = (char*)base;
  p.hdr = (CacheHeader*)b;
  p.m_prev = (float*)(b + align_up((size_t)n_req * sizeof(CacheHeader)));
  p.R = (float*)((char*)p.m_prev + align_up((size_t)tokens * c.hidden * 4));
  return p;
}

// Cache check on x0 (already embedded) with modulation rows set in P.
t2i_status cache_check_impl(t2i_dit* h, const Plan& P, int step, int n_steps, double tau,
                            int mode, void* state, double* rel_l1, uint8_t* skip, hipStream_t st) {
  const t2i_dit_config& c = h->cfg;
  CachePtrs cp = cache_ptrs(c, state, P.n_req, P.T_img);
  double* partial = h->at<double>(h->L.partial);
  // block 0's first LN-modulation (MMDiT: of the image stream)
  const int sh = is_mmdit(h) ? 6 * c.hidden : 0;
  HIP_TRY(h, prof_mark(h, T2I_K_CACHE, true, st));
  HIP_TRY(h, launch_cache_signal(h->at<float>(h->L.x0), P.rm, h->at<float>(h->L.mod),
                                 mod_width(c), sh, sh + c.hidden, c.hidden, c.ln_eps, cp.m_prev,
                                 cp.hdr, step, partial, st));
  HIP_TRY(h, launch_cache_decide(P.rm, partial, cp.hdr, step, n_steps, tau, mode, st));
  HIP_TRY(h, prof_mark(h, T2I_K_CACHE, false, st));
  h->hdr_host.resize(P.n_req);
  HIP_TRY(h, hipMemcpyAsync(h->hdr_host.data(), cp.hdr, sizeof(CacheHeader) * P.n_req,
                            hipMemcpyDeviceToHost, st));
  HIP_TRY(h, hipStreamSynchronize(st));
  for (int r = 0; r < P.n_req; ++r) {
    if (rel_l1) rel_l1[r] = h->hdr_host[r].d;
    if (skip) skip[r] = (uint8_t)(h->hdr_host[r].skip ? 1 : 0);
  }
  return T2I_OK;
}

// Packed byte offsets of one block's tensors (every block has the same
// shapes); returns the record size.
size_t block_layout(const t2i_dit_config& c, std::vector<size_t>* offs) {
  const std::vector<WDesc> t = weight_table(c);
  const size_t A = c.dtype == T2I_BF16 ? 2 : 4;
  size_t off = 0;
  for (int j = 0; j < per_block(c); ++j) {
    const WDesc& d = t[W_BLOCK0 + j];
    size_t n = 1;
    for (int k = 0; k < d.nd; ++k) n *= (size_t)d.shape[k];
    if (offs) offs->push_back(off);
    off = align_up(off + n * A);
  }
  return off;
}

// Loading blocks whose copy has finished become resident.
t2i_status refresh_loads(t2i_dit* h) {
  for (size_t b = 0; b < h->blk.size(); ++b) {
    if (h->blk[b] != t2i_dit::BLK_LOADING) continue;
    hipError_t e = hipEventQuery(h->blk_ev[b]);
    if (e == hipSuccess) h->blk[b] = t2i_dit::BLK_RESIDENT;
    else if (e != hipErrorNotReady)
      return fail(h, T2I_ERR_DEVICE, std::string("hipEventQuery: ") + hipGetErrorString(e));
  }
  return T2I_OK;
}

// Blocks [0, nb) must be resident or loading; the first still loading
// becomes P.defer_from.
t2i_status check_residency(t2i_dit* h, Plan& P, int nb) {
  if (t2i_status s = refresh_loads(h)) return s;
  P.defer_from = INT_MAX;
  for (int b = 0; b < nb; ++b) {
    if (h->blk[b] == t2i_dit::BLK_EVICTED)
      return fail(h, T2I_ERR_INVALID_ARG,
                  "block " + std::to_string(b) + " is evicted: queue its load first");
    if (h->blk[b] == t2i_dit::BLK_LOADING && P.defer_from == INT_MAX) P.defer_from = b;
  }
  return T2I_OK;
}

// Wait for every queued load (before the host tier or the bindings change).
t2i_status drain_loads(t2i_dit* h) {
  for (size_t b = 0; b < h->blk.size(); ++b)
    if (h->blk[b] == t2i_dit::BLK_LOADING) {
      HIP_TRY(h, hipEventSynchronize(h->blk_ev[b]));
      h->blk[b] = t2i_dit::BLK_RESIDENT;
    }
  return T2I_OK;
}

// The plan restricted to the requests in `mask`: their image rows packed in
// the same branch-major order; latent offsets, modulation rows and text rows
// (per request, plus the shared unconditional prompt) stay those of P, so the
// blocks compute for each of them exactly what they compute in P.  `g`
// receives the row segments that move P's layout to the compacted one.
void compute_subplan(const t2i_dit* h, const Plan& P, uint32_t mask, Plan& Q, RowCopyMap& g) {
  const int M = h->cfg.text_tokens;
  Q = P;
  int orig[kMaxReq];
  int n = 0, tok = 0;
  for (int r = 0; r < P.n_req; ++r) {
    if (!((mask >> r) & 1u)) continue;
    orig[n] = r;
    Q.rm.tok_off[n] = tok;
    Q.rm.lat_off[n] = P.rm.lat_off[r];
    Q.rm.h[n] = P.rm.h[r];
    Q.rm.w[n] = P.rm.w[r];
    Q.rm.modrow[n] = P.rm.modrow[r];
    Q.rm.dt[n] = P.rm.dt[r];
    tok += P.rm.tok_off[r + 1] - P.rm.tok_off[r];
    ++n;
  }
  Q.n_req = Q.rm.n = n;
  Q.rm.tok_off[n] = tok;
  Q.rm.tokens_total = Q.T_img = tok;
  Q.rows = tok * P.branches;
  Q.img.n = Q.self.n = Q.cross.n = n * P.branches;
  g.n = 0;
  int moved = 0;
  for (int br = 0; br < P.branches; ++br)
    for (int i = 0; i < n; ++i) {
      const int r = orig[i], s = br * n + i;
      const int start = br * tok + Q.rm.tok_off[i];
      const int len = Q.rm.tok_off[i + 1] - Q.rm.tok_off[i];
      Q.img.start[s] = start;
      Q.img.modrow[s] = P.rm.modrow[r];
      Q.self.q_start[s] = Q.cross.q_start[s] = start;
      Q.self.q_len[s] = Q.cross.q_len[s] = len;
      Q.self.k_start[s] = start;
      Q.self.k_len[s] = len;
      Q.cross.k_start[s] = br == 0 ? r * M : P.n_req * M;
      Q.cross.k_len[s] = M;
      g.src[g.n] = br * P.T_img + P.rm.tok_off[r];
      g.dst[g.n] = start;
      moved += len;
      g.row_end[g.n++] = moved;
    }
  Q.img.start[Q.img.n] = Q.rows;
  attention_tiles(Q.self, h->bf(), h->cfg.heads, 0);
  attention_tiles(Q.cross, h->bf(), h->cfg.heads, 1);
}

// Embed, blocks (or cached residual), final layer for one step whose
// conditioning rows start at `modbase`.
t2i_status step_body(t2i_dit* h, Plan& P, const float* latents_in, float* latents,
                     float* noise_pred, int nb, float* hidden_out, const uint8_t* skip,
                     void* cache_state, hipStream_t st) {
  const t2i_dit_config& c = h->cfg;
  const int D = c.hidden;
  float* x = h->at<float>(h->L.x);
  float* x0 = h->at<float>(h->L.x0);
  uint32_t skip_mask = 0, compute_mask = 0;
  for (int r = 0; r < P.n_req; ++r) {
    if (skip && skip[r]) skip_mask |= 1u << r;
    else compute_mask |= 1u << r;
  }
  // When some requests of a cross-DiT batch reuse their cached residual and
  // others compute, the blocks run on the computing requests' rows alone:
  // the call's image rows live in xf, the computing ones are gathered into
  // x, run, and scattered back.  (Not with a callback input, whose residuals
  // are laid out over every request.)
  const bool compact = skip_mask && compute_mask && nb > 0 && !is_mmdit(h) && !P.ctl &&
                       h->L.has_xf;
  float* xi = compact ? h->at<float>(h->L.xf)
                      : x + (size_t)img_row0(h, P) * D;   // image rows, the call's layout
  TIMED(h, T2I_K_EMBED, st, embed(h, P, latents_in, x0, xi, P.branches, st));
  if (is_mmdit(h))
    HIP_TRY(h, hipMemcpyAsync(x, h->at<float>(h->L.ytxt), (size_t)P.txt_rows * D * 4,
                              hipMemcpyDeviceToDevice, st));
  if (compact) {
    Plan Q;
    RowCopyMap g;
    compute_subplan(h, P, compute_mask, Q, g);
    HIP_TRY(h, launch_copy_rows(xi, x, g, D, st));
    t2i_status s = run_blocks(h, Q, nb, st);
    if (s != T2I_OK) return s;
    P.done = Q.done;
    RowCopyMap back = g;
    std::swap(back.src, back.dst);
    HIP_TRY(h, launch_copy_rows(x, xi, back, D, st));
  } else if (compute_mask) {
    t2i_status s = run_blocks(h, P, nb, st);
    if (s != T2I_OK) return s;
  }
  if (cache_state) {
    CachePtrs cp = cache_ptrs(c, cache_state, P.n_req, P.T_img);
    if (skip_mask) HIP_TRY(h, launch_apply_residual(x0, cp.R, xi, P.rm, skip_mask, D, st));
    if (compute_mask)
      HIP_TRY(h, launch_store_residual(x0, xi, cp.R, P.rm, compute_mask, D, cp.hdr, st));
  }
  if (hidden_out) {
    HIP_TRY(h, hipMemcpyAsync(hidden_out, xi, (size_t)P.rows * D * 4, hipMemcpyDeviceToDevice, st));
    if (is_mmdit(h))
      HIP_TRY(h, hipMemcpyAsync(hidden_out + (size_t)P.rows * D, x, (size_t)P.txt_rows * D * 4,
                                hipMemcpyDeviceToDevice, st));
  }
  const int mw = mod_width(c);
  const int fb = final_base(c);
  TIMED(h, T2I_K_FINAL, st,
        launch_final_layer(xi, P.rm, h->w[fb + 2], h->w[fb + 3], h->bf(), h->at<float>(h->L.mod),
                           mw, mw - 2 * D, mw - D, D, c.latent_channels, c.patch, c.ln_eps,
                           P.guidance, latents, noise_pred, st));
  return T2I_OK;
}

}  // namespace

// ===========================================================================
// exported

extern "C" {

const char* t2i_status_str(t2i_status s) {
  switch (s) {
    case T2I_OK: return "ok";
    case T2I_ERR_INVALID_ARG: return "invalid argument";
    case T2I_ERR_SHAPE: return "shape error";
    case T2I_ERR_UNSUPPORTED: return "unsupported";
    case T2I_ERR_WORKSPACE: return "workspace too small";
    case T2I_ERR_OUT_OF_MEMORY: return "out of memory";
    case T2I_ERR_DEVICE: return "device error";
  }
  return "unknown status";
}

const char* t2i_last_error(const t2i_dit* h) { return h ? h->err.c_str() : "NULL handle"; }

size_t t2i_dit_weight_count(const t2i_dit_config* cfg) {
  if (check_config(cfg)) return 0;
  return (size_t)final_base(*cfg) + 4;
}

t2i_status t2i_dit_weight_desc(const t2i_dit_config* cfg, size_t i, char name[64],
                               int64_t shape[4], int32_t* dtype) {
  if (check_config(cfg)) return T2I_ERR_INVALID_ARG;
  if (!name || !shape || !dtype) return T2I_ERR_INVALID_ARG;
  std::vector<WDesc> t = weight_table(*cfg);
  if (i >= t.size()) return T2I_ERR_SHAPE;
  std::snprintf(name, 64, "%s", t[i].name.c_str());
  for (int k = 0; k < 4; ++k) shape[k] = t[i].shape[k];
  *dtype = cfg->dtype;
  return T2I_OK;
}

size_t t2i_dit_workspace_bytes(const t2i_dit_config* cfg) {
  if (check_config(cfg)) return 0;
  return layout(*cfg).total;
}

size_t t2i_cache_state_bytes(const t2i_dit_config* cfg, int32_t n_req,
                             const int32_t* tokens_per_req, int32_t branches) {
  if (check_config(cfg) || n_req < 1 || n_req > cfg->max_requests || !tokens_per_req ||
      (branches != 1 && branches != 2))
    return 0;
  long tok = 0;
  for (int r = 0; r < n_req; ++r) {
    if (tokens_per_req[r] < 1) return 0;
    tok += tokens_per_req[r];
  }
  return cache_bytes(*cfg, n_req, (int)tok, branches);
}

t2i_status t2i_dit_init(const t2i_dit_config* cfg, const void* const* weights, void* workspace,
                        size_t ws_bytes, void* stream, t2i_dit** out) {
  (void)stream;
  if (!out) return T2I_ERR_INVALID_ARG;
  *out = nullptr;
  if (check_config(cfg)) return T2I_ERR_INVALID_ARG;
  if (!weights || !workspace) return T2I_ERR_INVALID_ARG;
  if ((uintptr_t)workspace % kAlign) return T2I_ERR_INVALID_ARG;
  const size_t need = layout(*cfg).total;
  if (ws_bytes < need) return T2I_ERR_WORKSPACE;
  const size_t n = (size_t)final_base(*cfg) + 4;
  for (size_t i = 0; i < n; ++i)
    if (!weights[i]) return T2I_ERR_INVALID_ARG;
  t2i_dit* h = new (std::nothrow) t2i_dit();
  if (!h) return T2I_ERR_OUT_OF_MEMORY;
  h->cfg = *cfg;
  h->w.assign(weights, weights + n);
  h->ws = (char*)workspace;
  h->ws_bytes = ws_bytes;
  h->L = layout(*cfg);
  h->blk.assign(cfg->depth, t2i_dit::BLK_RESIDENT);
  *out = h;
  return T2I_OK;
}

t2i_status t2i_dit_rebind_weights(t2i_dit* h, const void* const* weights, void* stream) {
  (void)stream;
  if (!h || !weights) return T2I_ERR_INVALID_ARG;
  for (size_t i = 0; i < h->w.size(); ++i)
    if (!weights[i]) return fail(h, T2I_ERR_INVALID_ARG, "NULL weight pointer");
  if (t2i_status s = drain_loads(h)) return s;
  h->w.assign(weights, weights + h->w.size());
  h->blk.assign(h->cfg.depth, t2i_dit::BLK_RESIDENT);
  return T2I_OK;
}

size_t t2i_dit_block_layout(const t2i_dit_config* cfg, int32_t* first_index, int32_t* n_tensors,
                            size_t* offsets) {
  if (check_config(cfg) || !first_index || !n_tensors) return 0;
  std::vector<size_t> o;
  const size_t bytes = block_layout(*cfg, &o);
  *first_index = W_BLOCK0;
  *n_tensors = per_block(*cfg);
  if (offsets) std::copy(o.begin(), o.end(), offsets);
  return bytes;
}

t2i_status t2i_dit_host_tier(t2i_dit* h, const void* host_blocks, void* arena,
                             size_t arena_bytes) {
  if (!h) return T2I_ERR_INVALID_ARG;
  if (!host_blocks || !arena) return fail(h, T2I_ERR_INVALID_ARG, "host_blocks and arena are required");
  if ((uintptr_t)arena % kAlign) return fail(h, T2I_ERR_INVALID_ARG, "arena must be 256-byte aligned");
  std::vector<size_t> offs;
  const size_t bb = block_layout(h->cfg, &offs);
  const size_t need = bb * (size_t)h->cfg.depth;
  if (arena_bytes < need) return fail(h, T2I_ERR_WORKSPACE, "arena smaller than depth * block_bytes");
  // both ends of each range must lie in memory of the right kind
  const char* hb = (const char*)host_blocks;
  const char* ab = (const char*)arena;
  const struct { const char* p; hipMemoryType want; const char* msg; } probes[] = {
      {hb, hipMemoryTypeHost, "host_blocks is not page-locked host memory"},
      {hb + need - 1, hipMemoryTypeHost, "host_blocks is not page-locked host memory"},
      {ab, hipMemoryTypeDevice, "arena is not device memory"},
      {ab + need - 1, hipMemoryTypeDevice, "arena is not device memory"}};
  for (const auto& pr : probes) {
    hipPointerAttribute_t at;
    std::memset(&at, 0, sizeof(at));
    hipError_t e = hipPointerGetAttributes(&at, pr.p);
    if (e != hipSuccess || at.type != pr.want) {
      (void)hipGetLastError();
      return fail(h, T2I_ERR_INVALID_ARG, pr.msg);
    }
  }
  if (t2i_status s = drain_loads(h)) return s;
  h->host_blocks = hb;
  h->arena = (char*)arena;
  h->blk_bytes = bb;
  h->blk_off = offs;
  return T2I_OK;
}

t2i_status t2i_dit_evict(t2i_dit* h, int32_t keep) {
  if (!h) return T2I_ERR_INVALID_ARG;
  if (!h->host_blocks) return fail(h, T2I_ERR_INVALID_ARG, "evict needs a host tier");
  const int depth = h->cfg.depth, pb = per_block(h->cfg);
  if (keep < 0 || keep > depth) return fail(h, T2I_ERR_SHAPE, "keep out of [0, depth]");
  for (int b = depth - 1; b >= keep; --b) {
    if (h->blk[b] == t2i_dit::BLK_LOADING) HIP_TRY(h, hipEventSynchronize(h->blk_ev[b]));
    h->blk[b] = t2i_dit::BLK_EVICTED;
    for (int j = 0; j < pb; ++j) h->w[W_BLOCK0 + (size_t)b * pb + j] = nullptr;
  }
  return T2I_OK;
}

t2i_status t2i_dit_load_async(t2i_dit* h, void* copy_stream, int32_t* n_loaded) {
  if (!h) return T2I_ERR_INVALID_ARG;
  if (n_loaded) *n_loaded = 0;
  if (!h->host_blocks) return fail(h, T2I_ERR_INVALID_ARG, "load needs a host tier");
  const int depth = h->cfg.depth, pb = per_block(h->cfg);
  hipStream_t cs = (hipStream_t)copy_stream;
  if (h->blk_ev.empty()) h->blk_ev.assign(depth, nullptr);
  int n = 0;
  for (int b = 0; b < depth; ++b) {
    if (h->blk[b] != t2i_dit::BLK_EVICTED) continue;
    if (!h->blk_ev[b])
      HIP_TRY(h, hipEventCreateWithFlags(&h->blk_ev[b], hipEventDisableTiming));
    char* dst = h->arena + (size_t)b * h->blk_bytes;
    HIP_TRY(h, hipMemcpyAsync(dst, h->host_blocks + (size_t)b * h->blk_bytes, h->blk_bytes,
                              hipMemcpyHostToDevice, cs));
    HIP_TRY(h, hipEventRecord(h->blk_ev[b], cs));
    for (int j = 0; j < pb; ++j) h->w[W_BLOCK0 + (size_t)b * pb + j] = dst + h->blk_off[j];
    h->blk[b] = t2i_dit::BLK_LOADING;
    ++n;
  }
  if (n_loaded) *n_loaded = n;
  return T2I_OK;
}

int32_t t2i_first_layers(int32_t L, double t_load, double t_comp) {
  if (L < 1 || !std::isfinite(t_load) || !std::isfinite(t_comp) || !(t_load > 0.0) ||
      !(t_comp > 0.0))
    return -1;
  // loading is hidden when the last copy, finished at (L - Le) t_load, still
  // leaves the last layer's compute as the only exposed time
  auto hides = [&](long le) { return (double)(L - le) * t_load + t_comp <= (double)L * t_comp; };
  const double v = std::ceil(((double)L * (t_load - t_comp) + t_comp) / t_load);
  long k = v < 1.0 ? 1 : v > (double)L ? L : (long)v;
  while (k > 1 && hides(k - 1)) --k;   // rounding of the quotient
  while (k < L && !hides(k)) ++k;
  return (int32_t)k;
}

t2i_status t2i_dit_block_state(t2i_dit* h, int32_t* state) {
  if (!h || !state) return T2I_ERR_INVALID_ARG;
  if (t2i_status s = refresh_loads(h)) return s;
  for (size_t b = 0; b < h->blk.size(); ++b) state[b] = h->blk[b];
  return T2I_OK;
}

void t2i_dit_destroy(t2i_dit* h) { delete h; }

t2i_status t2i_dit_profile(t2i_dit* h, uint32_t class_mask) {
  if (!h) return T2I_ERR_INVALID_ARG;
  if (class_mask >> T2I_K_COUNT) return fail(h, T2I_ERR_INVALID_ARG, "bad class mask");
  h->prof_mask = class_mask;
  h->ev_used = 0;
  h->ev_pairs.clear();
  return T2I_OK;
}

t2i_status t2i_dit_profile_read(t2i_dit* h, int32_t cls, double* total_ms, int64_t* launches) {
  if (!h || !total_ms || !launches) return T2I_ERR_INVALID_ARG;
  if (cls < 0 || cls >= T2I_K_COUNT) return fail(h, T2I_ERR_INVALID_ARG, "bad kernel class");
  if (h->ev_used) HIP_TRY(h, hipEventSynchronize(h->ev_pool[h->ev_used - 1]));
  double tot = 0.0;
  int64_t n = 0;
  for (const auto& pr : h->ev_pairs) {
    if (pr.first != cls) continue;
    float ms = 0.f;
    HIP_TRY(h, hipEventElapsedTime(&ms, h->ev_pool[pr.second], h->ev_pool[pr.second + 1]));
    tot += ms;
    ++n;
  }
  *total_ms = tot;
  *launches = n;
  return T2I_OK;
}

t2i_status t2i_dit_step(t2i_dit* h, const t2i_step_args* a, void* stream) {
  if (!h) return T2I_ERR_INVALID_ARG;
  if (!a || a->struct_size != sizeof(t2i_step_args))
    return fail(h, T2I_ERR_INVALID_ARG, "step args NULL or struct_size mismatch");
  if (!a->t || !a->latents || !a->prompt_embeds)
    return fail(h, T2I_ERR_INVALID_ARG, "t, latents and prompt_embeds are required");
  const t2i_dit_config& c = h->cfg;
  Plan P;
  t2i_status s = build_plan(h, a->n_req, a->lat_h, a->lat_w, a->guidance, P);
  if (s != T2I_OK) return s;
  const int nb = a->n_blocks < 0 ? c.depth : a->n_blocks;
  if (nb > c.depth) return fail(h, T2I_ERR_SHAPE, "n_blocks > depth");
  if (const t2i_control* ctl = a->control_outputs) {
    if (ctl->struct_size != sizeof(t2i_control))
      return fail(h, T2I_ERR_INVALID_ARG, "control_outputs struct_size mismatch");
    if (ctl->n < 1 || ctl->n > T2I_MAX_CONTROL)
      return fail(h, T2I_ERR_SHAPE, "control_outputs: n out of range");
    if (!ctl->blocks || !ctl->residuals)
      return fail(h, T2I_ERR_INVALID_ARG, "control_outputs: blocks / residuals is NULL");
    for (int i = 0; i < ctl->n; ++i) {
      if (ctl->blocks[i] < 0 || ctl->blocks[i] >= nb || (i && ctl->blocks[i] <= ctl->blocks[i - 1]))
        return fail(h, T2I_ERR_SHAPE,
                    "control_outputs: blocks must increase strictly and lie below the blocks run");
      if (!ctl->residuals[i]) return fail(h, T2I_ERR_INVALID_ARG, "control_outputs: NULL residual");
    }
    P.ctl = ctl;
  }
  if (a->skip && !a->cache_state)
    return fail(h, T2I_ERR_INVALID_ARG, "skip decisions need cache_state");
  if (a->cache_state &&
      a->cache_state_bytes < cache_bytes(c, P.n_req, P.T_img, P.branches))
    return fail(h, T2I_ERR_WORKSPACE, "cache_state too small");
  for (int r = 0; r < P.n_req; ++r) {
    if (!std::isfinite(a->t[r])) return fail(h, T2I_ERR_INVALID_ARG, "t not finite");
    if (a->t_next) {
      if (!std::isfinite(a->t_next[r])) return fail(h, T2I_ERR_INVALID_ARG, "t_next not finite");
      P.rm.dt[r] = (float)(a->t_next[r] - a->t[r]);
    }
  }
  if ((s = check_residency(h, P, std::max(nb, 1))) != T2I_OK) return s;
  hipStream_t st = (hipStream_t)stream;
  set_modrows(P, 0);
  P.cond_rows = P.n_req;
  if ((s = conditioning(h, a->t, P.n_req, std::max(nb, 1), P.defer_from, st)) != T2I_OK) return s;
  if ((s = text_prep(h, P, a->prompt_embeds, nb, st)) != T2I_OK) return s;
  return step_body(h, P, a->latents, a->latents, a->noise_pred, nb, a->hidden_out, a->skip,
                   a->cache_state, st);
}

t2i_status t2i_cache_check(t2i_dit* h, const t2i_cache_args* a, void* stream) {
  if (!h) return T2I_ERR_INVALID_ARG;
  if (!a || a->struct_size != sizeof(t2i_cache_args))
    return fail(h, T2I_ERR_INVALID_ARG, "cache args NULL or struct_size mismatch");
  if (!a->t || !a->latents || !a->cache_state || !a->rel_l1 || !a->skip)
    return fail(h, T2I_ERR_INVALID_ARG, "missing pointer");
  if (a->step < 0 || a->step >= a->n_steps) return fail(h, T2I_ERR_SHAPE, "bad step");
  if (a->mode != T2I_CACHE_ACCUMULATE && a->mode != T2I_CACHE_PER_STEP)
    return fail(h, T2I_ERR_INVALID_ARG, "bad mode");
  if (a->branches != 1 && a->branches != 2) return fail(h, T2I_ERR_INVALID_ARG, "bad branches");
  Plan P;
  t2i_status s = build_plan(h, a->n_req, a->lat_h, a->lat_w, a->branches == 2 ? 2.f : 1.f, P);
  if (s != T2I_OK) return s;
  const t2i_dit_config& c = h->cfg;
  if (a->cache_state_bytes < cache_bytes(c, P.n_req, P.T_img, P.branches))
    return fail(h, T2I_ERR_WORKSPACE, "cache_state too small");
  if ((s = check_residency(h, P, 1)) != T2I_OK) return s;
  hipStream_t st = (hipStream_t)stream;
  set_modrows(P, 0);
  // block 0's modulation only: a loading block 0 is waited for in place
  if ((s = conditioning(h, a->t, P.n_req, 1, INT_MAX, st)) != T2I_OK) return s;
  HIP_TRY(h, embed(h, P, a->latents, h->at<float>(h->L.x0), h->at<float>(h->L.x), 0, st));
  return cache_check_impl(h, P, a->step, a->n_steps, a->tau, a->mode, a->cache_state, a->rel_l1,
                          a->skip, st);
}

t2i_status t2i_dit_sample(t2i_dit* h, const t2i_sample_args* a, void* stream) {
  if (!h) return T2I_ERR_INVALID_ARG;
  if (!a || a->struct_size != sizeof(t2i_sample_args))
    return fail(h, T2I_ERR_INVALID_ARG, "sample args NULL or struct_size mismatch");
  if (!a->latents || !a->prompt_embeds) return fail(h, T2I_ERR_INVALID_ARG, "missing pointer");
  const t2i_dit_config& c = h->cfg;
  if (a->n_steps < 1 || a->n_steps > c.max_steps) return fail(h, T2I_ERR_SHAPE, "n_steps out of range");
  if (a->start_step < 0 || a->start_step >= a->n_steps) return fail(h, T2I_ERR_SHAPE, "bad start_step");
  const bool use_cache = a->cache_tau > 0.0;
  if (use_cache && (!a->cache_state)) return fail(h, T2I_ERR_INVALID_ARG, "cache needs cache_state");
  if (a->cache_mode != T2I_CACHE_ACCUMULATE && a->cache_mode != T2I_CACHE_PER_STEP)
    return fail(h, T2I_ERR_INVALID_ARG, "bad cache_mode");
  Plan P;
  t2i_status s = build_plan(h, a->n_req, a->lat_h, a->lat_w, a->guidance, P);
  if (s != T2I_OK) return s;
  if (use_cache && a->cache_state_bytes < cache_bytes(c, P.n_req, P.T_img, P.branches))
    return fail(h, T2I_ERR_WORKSPACE, "cache_state too small");
  const int n = a->n_steps, R = P.n_req;
  std::vector<double> ts((size_t)(n + 1) * R);
  for (int k = 0; k <= n; ++k)
    for (int r = 0; r < R; ++r) {
      const double v = a->timesteps ? a->timesteps[(size_t)k * R + r] : 1.0 - (double)k / n;
      if (!std::isfinite(v)) return fail(h, T2I_ERR_INVALID_ARG, "timestep not finite");
      ts[(size_t)k * R + r] = v;
    }
  if ((s = check_residency(h, P, c.depth)) != T2I_OK) return s;
  hipStream_t st = (hipStream_t)stream;
  // conditioning rows k*R + r for every step k < n
  P.cond_rows = n * R;
  if ((s = conditioning(h, ts.data(), n * R, c.depth, P.defer_from, st)) != T2I_OK) return s;
  if ((s = text_prep(h, P, a->prompt_embeds, c.depth, st)) != T2I_OK) return s;
  std::vector<uint8_t> skip(R, 0);
  std::vector<double> rel(R, 0.0);
  for (int k = a->start_step; k < n; ++k) {
    set_modrows(P, k * R);
    for (int r = 0; r < R; ++r)
      P.rm.dt[r] = (float)(ts[(size_t)(k + 1) * R + r] - ts[(size_t)k * R + r]);
    if (use_cache) {
      HIP_TRY(h, embed(h, P, a->latents, h->at<float>(h->L.x0), h->at<float>(h->L.x), 0, st));
      if ((s = ensure_block(h, P, 0, st)) != T2I_OK) return s;   // block 0's modulation
      if ((s = cache_check_impl(h, P, k, n, a->cache_tau, a->cache_mode, a->cache_state,
                                rel.data(), skip.data(), st)) != T2I_OK)
        return s;
    }
    for (int r = 0; r < R; ++r) {
      if (a->skip_log) a->skip_log[(size_t)k * R + r] = skip[r];
      if (a->rel_l1_log) a->rel_l1_log[(size_t)k * R + r] = use_cache ? rel[r] : NAN;
    }
    if ((s = step_body(h, P, a->latents, a->latents, nullptr, c.depth, nullptr,
                       use_cache ? skip.data() : nullptr, use_cache ? a->cache_state : nullptr,
                       st)) != T2I_OK)
      return s;
  }
  return T2I_OK;
}

// ---------------------------------------------------------------------------
// kernel-level entry points

const char* t2i_ops_last_error(void) { return g_ops_err.c_str(); }

static t2i_status ops_fail(t2i_status s, const std::string& m) {
  g_ops_err = m;
  return s;
}

t2i_status t2i_op_linear(int32_t dtype, int32_t epilogue, int32_t M, int32_t N, int32_t K,
                         const void* A, int32_t lda, const void* W, int32_t ldw, const void* bias,
                         void* out, int32_t ldo, float* resid, int32_t ldr, void* resid_copy,
                         const float* gate, void* stream) {
  if (dtype != T2I_F32 && dtype != T2I_BF16) return ops_fail(T2I_ERR_INVALID_ARG, "bad dtype");
  if (epilogue < T2I_EPI_STORE || epilogue > T2I_EPI_RESID_GATED)
    return ops_fail(T2I_ERR_INVALID_ARG, "bad epilogue");
  if (M < 1 || N < 1 || K < 1) return ops_fail(T2I_ERR_SHAPE, "empty GEMM");
  if (!A || !W || !bias) return ops_fail(T2I_ERR_INVALID_ARG, "NULL operand");
  if (lda < K || ldw < K) return ops_fail(T2I_ERR_SHAPE, "leading dimension < K");
  const bool res = epilogue >= T2I_EPI_RESID;
  if (res && (!resid || ldr < N)) return ops_fail(T2I_ERR_INVALID_ARG, "bad residual");
  if (!res && (!out || ldo < N)) return ops_fail(T2I_ERR_INVALID_ARG, "bad out");
  if (epilogue == T2I_EPI_RESID_GATED && !gate) return ops_fail(T2I_ERR_INVALID_ARG, "NULL gate");
  if (dtype == T2I_BF16 && (K % 64 || lda % 8 || ldw % 8))
    return ops_fail(T2I_ERR_SHAPE, "bf16 GEMM needs K % 64 == 0 and lda, ldw % 8 == 0");
  Epi e = make_epi();
  e.out = out;
  e.ldo = ldo;
  e.x = resid;
  e.ldx = ldr;
  e.xb = (bf16*)resid_copy;
  e.gate = gate;
  e.ld_gate = 0;
  e.map.n = 1;
  e.map.start[0] = 0;
  e.map.start[1] = M;
  e.map.modrow[0] = 0;
  hipStream_t st = (hipStream_t)stream;
  hipError_t err = dtype == T2I_BF16
                       ? launch_gemm_bf16((const bf16*)A, lda, (const bf16*)W, ldw, (const bf16*)bias,
                                          M, N, K, epilogue, e, nullptr, 0, st)
                       : launch_gemm_f32((const float*)A, lda, W, ldw, false, bias, M, N, K,
                                         epilogue, e, st);
  if (err != hipSuccess) return ops_fail(T2I_ERR_DEVICE, hipGetErrorString(err));
  return T2I_OK;
}

t2i_status t2i_op_attention(int32_t dtype, int32_t heads, int32_t head_dim, int32_t n_seq,
                            const int32_t* q_start, const int32_t* q_len, const int32_t* k_start,
                            const int32_t* k_len, const int32_t* k2_start, const int32_t* k2_len,
                            const void* q, int32_t ldq, const void* k, int32_t ldk, const void* v,
                            int32_t ldv, void* o, int32_t ldo, void* stream) {
  if (dtype != T2I_F32 && dtype != T2I_BF16) return ops_fail(T2I_ERR_INVALID_ARG, "bad dtype");
  if (heads < 1 || (head_dim != 8 && head_dim != 32 && head_dim != 64 && head_dim != 72 &&
                    head_dim != 128))
    return ops_fail(T2I_ERR_SHAPE, "unsupported head_dim");
  if (n_seq < 1 || n_seq > kMaxSeq) return ops_fail(T2I_ERR_SHAPE, "bad n_seq");
  if (!q_start || !q_len || !k_start || !k_len || !q || !k || !v || !o)
    return ops_fail(T2I_ERR_INVALID_ARG, "NULL pointer");
  if (!k2_start != !k2_len) return ops_fail(T2I_ERR_INVALID_ARG, "k2_start and k2_len go together");
  const int w = heads * head_dim;
  if (ldq < w || ldk < w || ldo < w || ldq % 8 || ldk % 8 || ldv % 8 || ldo % 8 ||
      (dtype == T2I_F32 && ldv < w))
    return ops_fail(T2I_ERR_SHAPE, "bad leading dimension");
  AttnMap m;
  std::memset(&m, 0, sizeof(m));   // no second key segment
  m.n = n_seq;
  for (int s = 0; s < n_seq; ++s) {
    const int s2 = k2_start ? k2_start[s] : 0, n2 = k2_len ? k2_len[s] : 0;
    if (q_start[s] < 0 || q_len[s] < 0 || k_start[s] < 0 || k_len[s] < 0 || s2 < 0 || n2 < 0 ||
        k_len[s] + n2 < 1)
      return ops_fail(T2I_ERR_SHAPE, "bad sequence bounds");
    if (dtype == T2I_BF16 && (k_start[s] % 8 || (long)k_start[s] + k_len[s] > ldv || s2 % 8 ||
                              (long)s2 + n2 > ldv))
      return ops_fail(T2I_ERR_SHAPE, "bf16 attention needs key starts % 8 == 0 and keys within ldv");
    m.q_start[s] = q_start[s];
    m.q_len[s] = q_len[s];
    m.k_start[s] = k_start[s];
    m.k_len[s] = k_len[s];
    m.k2_start[s] = s2;
    m.k2_len[s] = n2;
  }
  if (dtype == T2I_BF16) {
    long k_rows = 0;
    for (int s = 0; s < n_seq; ++s)
      k_rows = std::max({k_rows, (long)k_start[s] + k_len[s],
                         k2_start ? (long)k2_start[s] + k2_len[s] : 0L});
    if ((size_t)2 * heads * head_dim * ldv > 0x7fffffff ||
        (size_t)2 * (k_rows + 64) * ldk > 0x7fffffff)
      return ops_fail(T2I_ERR_SHAPE, "bf16 attention operands exceed 2 GiB of addressing");
  }
  attention_tiles(m, dtype == T2I_BF16, heads, 0);
  hipError_t err = launch_attention(dtype == T2I_BF16, 0, heads, head_dim, m, q, ldq, k, ldk, v, ldv,
                                    o, ldo, (hipStream_t)stream, false);
  if (err != hipSuccess) return ops_fail(T2I_ERR_DEVICE, hipGetErrorString(err));
  return T2I_OK;
}

t2i_status t2i_op_cross_attention(int32_t dtype, int32_t heads, int32_t head_dim, int32_t n_seq,
                                  const int32_t* q_start, const int32_t* q_len,
                                  const int32_t* k_start, const int32_t* k_len, const void* q,
                                  int32_t ldq, const void* k, int32_t ldk, const void* v,
                                  int32_t ldv, void* o, int32_t ldo, void* stream) {
  if (dtype != T2I_BF16) return ops_fail(T2I_ERR_INVALID_ARG, "cross-attention is bf16 only");
  if (heads < 1 || (head_dim != 8 && head_dim != 32 && head_dim != 64 && head_dim != 72 &&
                    head_dim != 128))
    return ops_fail(T2I_ERR_SHAPE, "unsupported head_dim");
  if (n_seq < 1 || n_seq > kMaxSeq) return ops_fail(T2I_ERR_SHAPE, "bad n_seq");
  if (!q_start || !q_len || !k_start || !k_len || !q || !k || !v || !o)
    return ops_fail(T2I_ERR_INVALID_ARG, "NULL pointer");
  const int w = heads * head_dim;
  if (ldq < w || ldk < w || ldo < w || ldq % 8 || ldk % 8 || ldv % 8 || ldo % 8)
    return ops_fail(T2I_ERR_SHAPE, "bad leading dimension");
  AttnMap m;
  std::memset(&m, 0, sizeof(m));
  m.n = n_seq;
  long k_rows = 0;
  for (int s = 0; s < n_seq; ++s) {
    if (q_start[s] < 0 || q_len[s] < 0 || k_start[s] < 0 || k_len[s] < 1)
      return ops_fail(T2I_ERR_SHAPE, "bad sequence bounds");
    if (k_start[s] % 8 || (long)k_start[s] + k_len[s] > ldv)
      return ops_fail(T2I_ERR_SHAPE, "bf16 attention needs key starts % 8 == 0 and keys within ldv");
    m.q_start[s] = q_start[s];
    m.q_len[s] = q_len[s];
    m.k_start[s] = k_start[s];
    m.k_len[s] = k_len[s];
    k_rows = std::max(k_rows, (long)k_start[s] + k_len[s]);
  }
  if ((size_t)2 * heads * head_dim * ldv > 0x7fffffff || (size_t)2 * (k_rows + 64) * ldk > 0x7fffffff)
    return ops_fail(T2I_ERR_SHAPE, "bf16 attention operands exceed 2 GiB of addressing");
  attention_tiles(m, true, heads, 1);
  hipError_t err = launch_attention(true, 1, heads, head_dim, m, q, ldq, k, ldk, v, ldv, o, ldo,
                                    (hipStream_t)stream, false);
  if (err != hipSuccess) return ops_fail(T2I_ERR_DEVICE, hipGetErrorString(err));
  return T2I_OK;
}

t2i_status t2i_op_linear_cross_attention(int32_t fused, int32_t heads, int32_t head_dim,
                                         int32_t n_seq, const int32_t* q_start,
                                         const int32_t* q_len, const int32_t* k_start,
                                         const int32_t* k_len, int32_t K, const void* A,
                                         int32_t lda, const void* W, int32_t ldw, const void* bias,
                                         const void* k, int32_t ldk, const void* v, int32_t ldv,
                                         void* q_buf, int32_t ldq, void* o, int32_t ldo,
                                         void* stream) {
  if (fused != 0 && fused != 1) return ops_fail(T2I_ERR_INVALID_ARG, "fused must be 0 or 1");
  if (heads < 1 || (head_dim != 8 && head_dim != 32 && head_dim != 64 && head_dim != 72 &&
                    head_dim != 128))
    return ops_fail(T2I_ERR_SHAPE, "unsupported head_dim");
  if (n_seq < 1 || n_seq > kMaxSeq) return ops_fail(T2I_ERR_SHAPE, "bad n_seq");
  if (!q_start || !q_len || !k_start || !k_len || !A || !W || !bias || !k || !v || !o)
    return ops_fail(T2I_ERR_INVALID_ARG, "NULL pointer");
  if (!fused && !q_buf) return ops_fail(T2I_ERR_INVALID_ARG, "NULL q_buf (needed when fused == 0)");
  const int w = heads * head_dim;
  if (K < 64 || K % 64 || lda < K || ldw < K || lda % 8 || ldw % 8)
    return ops_fail(T2I_ERR_SHAPE, "bf16 GEMM needs K % 64 == 0 and lda, ldw >= K, % 8 == 0");
  if (ldk < w || ldo < w || ldk % 8 || ldv % 8 || ldo % 8 || (!fused && (ldq < w || ldq % 8)))
    return ops_fail(T2I_ERR_SHAPE, "bad leading dimension");
  AttnMap m;
  std::memset(&m, 0, sizeof(m));
  m.n = n_seq;
  long k_rows = 0;
  int M = 0;
  for (int s = 0; s < n_seq; ++s) {
    if (q_start[s] < 0 || q_len[s] < 0 || k_start[s] < 0 || k_len[s] < 1 || k_len[s] > 128)
      return ops_fail(T2I_ERR_SHAPE, "bad sequence bounds (text of 1 .. 128 keys)");
    if (k_start[s] % 8 || (long)k_start[s] + k_len[s] > ldv)
      return ops_fail(T2I_ERR_SHAPE, "bf16 attention needs key starts % 8 == 0 and keys within ldv");
    m.q_start[s] = q_start[s];
    m.q_len[s] = q_len[s];
    m.k_start[s] = k_start[s];
    m.k_len[s] = k_len[s];
    k_rows = std::max(k_rows, (long)k_start[s] + k_len[s]);
    M = std::max(M, q_start[s] + q_len[s]);
  }
  if (M < 1) return ops_fail(T2I_ERR_SHAPE, "no query rows");
  if ((size_t)2 * heads * head_dim * ldv > 0x7fffffff || (size_t)2 * (k_rows + 64) * ldk > 0x7fffffff)
    return ops_fail(T2I_ERR_SHAPE, "bf16 attention operands exceed 2 GiB of addressing");
  // the query projection's epilogue: softmax scale folded in, one rounding
  Epi e = make_epi();
  e.out = q_buf;
  e.ldo = ldq;
  e.qscale = attn_q_scale(head_dim);
  e.qcols = w;
  hipStream_t st = (hipStream_t)stream;
  hipError_t err;
  if (fused) {
    const XAttnArgs xa = make_xattn(m, k, ldk, v, ldv, o, ldo);
    err = launch_gemm_xattn((const bf16*)A, lda, (const bf16*)W, ldw, (const bf16*)bias, M, w, K, e,
                            heads, head_dim, xa, st, true);
    if (err == hipErrorNotSupported)
      return ops_fail(T2I_ERR_SHAPE,
                      "shapes outside the fused kernel (head_dim 72, K % 192 == 0, sequences "
                      "contiguous from row 0 with lengths % 256 == 0, 16-byte aligned operands)");
    if (err == hipSuccess)
      err = launch_gemm_xattn((const bf16*)A, lda, (const bf16*)W, ldw, (const bf16*)bias, M, w, K,
                              e, heads, head_dim, xa, st);
  } else {
    err = launch_gemm_bf16((const bf16*)A, lda, (const bf16*)W, ldw, (const bf16*)bias, M, w, K,
                           EPI_STORE, e, nullptr, 0, st);
    if (err == hipSuccess) {
      attention_tiles(m, true, heads, 1);
      err = launch_attention(true, 1, heads, head_dim, m, q_buf, ldq, k, ldk, v, ldv, o, ldo, st,
                             true);
    }
  }
  if (err != hipSuccess) return ops_fail(T2I_ERR_DEVICE, hipGetErrorString(err));
  return T2I_OK;
}

t2i_status t2i_op_ln_modulate(int32_t dtype, int32_t rows, int32_t D, const float* x,
                              const float* shift, const float* scale, float eps, void* out,
                              void* stream) {
  if (dtype != T2I_F32 && dtype != T2I_BF16) return ops_fail(T2I_ERR_INVALID_ARG, "bad dtype");
  if (rows < 1 || D < 4 || D % 4 || D > 3072) return ops_fail(T2I_ERR_SHAPE, "bad shape");
  if (!x || !shift || !scale || !out) return ops_fail(T2I_ERR_INVALID_ARG, "NULL pointer");
  if (scale != shift + D) return ops_fail(T2I_ERR_INVALID_ARG, "scale must follow shift (scale == shift + D)");
  if ((uintptr_t)x % 16 || (uintptr_t)shift % 16 || (uintptr_t)out % (dtype == T2I_BF16 ? 8 : 16))
    return ops_fail(T2I_ERR_INVALID_ARG, "x, shift need 16-byte and out 8 (bf16) / 16-byte alignment");
  SeqMap m;
  std::memset(&m, 0, sizeof(m));
  m.n = 1;
  m.start[1] = rows;
  hipError_t err = launch_ln_modulate(dtype == T2I_BF16, rows, D, x, D, shift, 2 * D, 0, D, m, out,
                                      D, eps, (hipStream_t)stream);
  if (err != hipSuccess) return ops_fail(T2I_ERR_DEVICE, hipGetErrorString(err));
  return T2I_OK;
}

t2i_status t2i_op_lora_merge_batch(int32_t dtype, int32_t n, int32_t n_out, int32_t n_in,
                                   int32_t rank, float alpha, void* const* W, int32_t ldw,
                                   const void* const* A, const void* const* B, void* stream) {
  if (dtype != T2I_F32 && dtype != T2I_BF16) return ops_fail(T2I_ERR_INVALID_ARG, "bad dtype");
  if (n < 1) return ops_fail(T2I_ERR_SHAPE, "n must be >= 1");
  if (n_out < 1 || n_in < 1 || ldw < n_in) return ops_fail(T2I_ERR_SHAPE, "bad weight shape");
  if (rank < 1 || rank > 128) return ops_fail(T2I_ERR_SHAPE, "rank must be in 1 .. 128");
  if (!W || !A || !B) return ops_fail(T2I_ERR_INVALID_ARG, "NULL pointer table");
  for (int i = 0; i < n; ++i)
    if (!W[i] || !A[i] || !B[i]) return ops_fail(T2I_ERR_INVALID_ARG, "NULL pointer");
  if (!std::isfinite(alpha)) return ops_fail(T2I_ERR_INVALID_ARG, "alpha not finite");
  for (int i0 = 0; i0 < n; i0 += kMaxGroups) {
    LoraGroup g;
    const int m = std::min(kMaxGroups, n - i0);
    for (int i = 0; i < m; ++i) {
      g.W[i] = W[i0 + i];
      g.A[i] = A[i0 + i];
      g.B[i] = B[i0 + i];
    }
    hipError_t err = launch_lora_merge_group(dtype == T2I_BF16, m, n_out, n_in, rank, alpha, g,
                                             ldw, (hipStream_t)stream);
    if (err != hipSuccess) return ops_fail(T2I_ERR_DEVICE, hipGetErrorString(err));
  }
  return T2I_OK;
}

t2i_status t2i_op_dma_read(const void* src, size_t bytes, float* sink, void* stream) {
  if (!src || !sink) return ops_fail(T2I_ERR_INVALID_ARG, "NULL pointer");
  if (bytes == 0 || bytes % 1024 || bytes > ((size_t)1 << 31) - 1024)
    return ops_fail(T2I_ERR_SHAPE, "bytes must be a positive multiple of 1024 below 2 GiB");
  if ((uintptr_t)src % 16) return ops_fail(T2I_ERR_INVALID_ARG, "src must be 16-byte aligned");
  hipError_t err = launch_dma_read(src, bytes, sink, (hipStream_t)stream);
  if (err != hipSuccess) return ops_fail(T2I_ERR_DEVICE, hipGetErrorString(err));
  return T2I_OK;
}

t2i_status t2i_op_lora_merge(int32_t dtype, int32_t n_out, int32_t n_in, int32_t rank,
                             float alpha, void* W, int32_t ldw, const void* A, const void* B,
                             void* stream) {
  if (dtype != T2I_F32 && dtype != T2I_BF16) return ops_fail(T2I_ERR_INVALID_ARG, "bad dtype");
  if (n_out < 1 || n_in < 1 || ldw < n_in) return ops_fail(T2I_ERR_SHAPE, "bad weight shape");
  if (rank < 1 || rank > 128) return ops_fail(T2I_ERR_SHAPE, "rank must be in 1 .. 128");
  if (!W || !A || !B) return ops_fail(T2I_ERR_INVALID_ARG, "NULL pointer");
  if (!std::isfinite(alpha)) return ops_fail(T2I_ERR_INVALID_ARG, "alpha not finite");
  hipError_t err = launch_lora_merge(dtype == T2I_BF16, n_out, n_in, rank, alpha, W, ldw, A, B,
                                     (hipStream_t)stream);
  if (err != hipSuccess) return ops_fail(T2I_ERR_DEVICE, hipGetErrorString(err));
  return T2I_OK;
}

}  // extern "C"
