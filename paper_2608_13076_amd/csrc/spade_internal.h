// Internal declarations shared by the C ABI (api.cpp) and the kernels
// (kernels.hip).  Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/spade.h"

namespace spade {

constexpr int kPanel = 16;           // weight rows per MFMA tile (one panel)
constexpr int kTileBytes = 8192;     // one panel x one k-block, in the arena
constexpr int kMaxRowsPerGemm = 32;  // rows handled by one skinny-GEMM launch
constexpr int kWideMinRows = 16;     // bf16 projections with more rows use the wide-row GEMM
constexpr int kPrefillRows = 16;     // prompt rows per request of a prefill forward on the verify attention
constexpr int kPrefillMaxRows = 2048;  // rows of a prefill forward (bf16 cache, head_dim 128)
constexpr int kPrefillAttnTiles = 4;   // 16-row tiles (one wave each) per workgroup of the prefill attention
constexpr int kPrefillAttnKeys = 64;   // keys per K or V^T block it stages in LDS
constexpr int kMaxR = 16;            // rows per request in one forward (gamma <= 15)
constexpr int kCorrMaxSlices = 256; // vocabulary slices of one correction draw
constexpr int kNoAllocMaxB = 64;     // requests of one spade_accept_from_logits_noalloc call
constexpr int kActSplits = 2;        // bf16 terms per fp32 activation (hi, lo)
constexpr int kAttnChunk = 128;      // keys per workgroup of the generic attention (f32 cache or head_dim != 128)
constexpr int kAttnMaxChunks = 128;  // chunks per (request, head)
constexpr int kMaxLen = kAttnChunk * kAttnMaxChunks;
constexpr int kMaxStatGroups = 2048;             // LM-head statistics entries per row (workgroups)
// The V cache is stored in blocks of kVBlock positions (head_dim x kVBlock
// elements, one contiguous run per (request, K/V head)); positions per
// (request, K/V head) of either cache: max_len rounded up to a whole block.
constexpr int kVBlock = 256;
inline int kv_stride_of(int max_len) { return (max_len + kVBlock - 1) / kVBlock * kVBlock; }
// Element (feature f, position pos) of a (request, K/V head) V region of a
// bf16 cache: a block is the B operands of O = P V in MFMA order, fragment
// (16-feature tile f / 16, 32-position step p / 32) of 1 KB, whose lane
// 16 ((p / 8) % 4) + f % 16 holds positions 8 ((p / 8) % 4) .. + 7 of the step
// (p = pos % kVBlock), so one wave's fragment load reads 1 KB contiguous.
__host__ __device__ inline size_t v_cache_index(int f, int pos, int hd) {
  const int p = pos % kVBlock;
  return (size_t)(pos / kVBlock) * hd * kVBlock +
         (size_t)(((((f >> 4) * (kVBlock / 32) + (p >> 5)) * 64 + ((p >> 3) & 3) * 16 + (f & 15)) * 8) + (p & 7));
}
// ... and of a float32 cache: a block is [head_dim][kVBlock].
__host__ __device__ inline size_t v_cache_index_f32(int f, int pos, int hd) {
  return ((size_t)(pos / kVBlock) * hd + f) * kVBlock + (pos % kVBlock);
}
// Element (feature f, position pos) of a (request, K/V head) K region of a
// bf16 cache, in blocks of kVBlock positions: a block is the B operands of
// S = Q K^T in MFMA order, fragment (16-position group p / 16, 32-feature
// step f / 32) of 1 KB, whose lane 16 ((f / 8) % 4) + p % 16 holds features
// 8 ((f / 8) % 4) .. + 7 of position p (p = pos % kVBlock), so one wave's
// fragment load reads 1 KB contiguous.  A float32 K cache is [position][head_dim].
__host__ __device__ inline size_t k_cache_index(int f, int pos, int hd) {
  const int p = pos % kVBlock;
  return (size_t)(pos / kVBlock) * hd * kVBlock +
         (size_t)(((((p >> 4) * (hd >> 5) + (f >> 5)) * 64 + ((f >> 3) & 3) * 16 + (p & 15)) * 8) + (f & 7));
}

// Keys per chunk of the bf16 / head_dim-128 verify attention.  A constant:
// a request's attention (and so its logits) must not depend on the other
// requests of the batch.  256 keys: 78 VGPRs and 35 KB of LDS per 8-wave
// workgroup of the one-chunk kernel, three workgroups per compute unit.
constexpr int kAttnChunkKeys = 256;
constexpr int kAttnHd = 128;  // head_dim of the MFMA attention kernels (bf16 cache)

enum GemmKind { GEMM_QKV = 0, GEMM_O = 1, GEMM_GU = 2, GEMM_DOWN = 3, GEMM_LM = 4 };

inline int kblock_of(int weight_dtype) { return weight_dtype == SPADE_BF16 ? 256 : 128; }

// QKV section of arena panel p: 0 (queries, d_model / 16 panels), 1 (keys) or
// 2 (values, dkv / 16 panels each), and the panel's index within it.
__host__ __device__ inline int qkv_section(int p, int d_model, int dkv, int* pw) {
  const int pq = d_model / 16, pk = dkv / 16;
  const int s = p < pq ? 0 : (p < pq + pk ? 1 : 2);
  *pw = p - (s == 0 ? 0 : (s == 1 ? pq : pq + pk));
  return s;
}

// Row of the logical [N, K] weight matrix held by row r (0..15) of arena
// panel p.  Panels are stored in order, each as its k-blocks in order.
//   QKV (N = d + 2 dkv, rows of Wq, Wk, Wv; dkv = kv heads * hd): panel p of
//     section s holds, for head h and group w, features w*8 .. w*8+7 in rows
//     0..7 and their rotary partners w*8+hd/2 .. w*8+7+hd/2 in rows 8..15, so
//     lanes n and n^8 of an MFMA output hold a RoPE pair.
//   GU (N = 2F, gate rows then up rows): panel p holds gate rows p*8 .. p*8+7
//     in rows 0..7 and the matching up rows in rows 8..15.
//   O, DOWN, LM: panel p holds rows p*16 .. p*16+15.
__host__ __device__ inline int panel_row(int kind, int p, int r, int d_model, int head_dim, int d_ffn, int dkv) {
  if (kind == GEMM_QKV) {
    const int pph = head_dim / 16;
    int pw;
    const int s = qkv_section(p, d_model, dkv, &pw);
    const int h = pw / pph, w = pw % pph;
    const int f = w * 8 + (r & 7) + (r >= 8 ? head_dim / 2 : 0);
    return (s == 0 ? 0 : (s == 1 ? d_model : d_model + dkv)) + h * head_dim + f;
  }
  if (kind == GEMM_GU) return (r < 8) ? p * 8 + r : d_ffn + p * 8 + (r - 8);
  return p * 16 + r;
}

struct Dims {
  int L, d, H, hd, F, V, Vpad, wdt, kvdt;
  int KVH, dkv;  // K/V heads (grouped-query attention: H / KVH query heads each) and their width KVH * hd
  float eps, theta;
};

// Byte offsets of every tensor inside the weight arena.
struct ArenaLayout {
  size_t qkv, o, gu, down, g_attn, g_ffn;  // per-layer offsets relative to layer base
  size_t layer_bytes;
  size_t embed, g_final, lm, total;
};

// Sub-buffers of the caller's workspace.
struct Workspace {
  float* x;           // [Mrows][d] residual stream
  void* act_n;        // normed GEMM input, split bf16 [S][Mrows][d] or f32 [Mrows][d]
  void* act_o;        // attention output (O-projection input)
  void* act_f;        // SwiGLU output (down-projection input) [S][Mrows][F]
  float* ssq;         // [Mrows][d/16] sum-of-squares partials of x
  float* q;           // [Mrows][d] rotated queries
  float* attn_o;      // [Bmax][H][NCmax][Rmax][hd] chunk partial outputs
  float* attn_ml;     // [Bmax][H][NCmax][Rmax][2] chunk max / sum
  uint32_t* attn_cnt; // [Bmax][H] arrival counters (kept at zero between calls)
  float* logits;      // [Mmax][V]
  float* stats;       // [Mmax][groups][3] LM-head per-workgroup max / sumexp / argmax
  float* rope;        // [max_len][hd/2][2] cos, sin
  uint32_t* err;      // device error word
  uint32_t* split_cnt;  // [max units / 2] arrival counters of the split-K GEMM (kept at zero between calls)
  float* split_part;    // [max units][8][256] published sums and range partials of the split-K GEMM
  uint32_t* wide_cnt;   // [wide_items] arrival counters of the k-split wide-row GEMM (kept at zero between calls)
  float* wide_part;     // [wide_floats] its published sums and range partials
  size_t wide_items, wide_floats;
  float* mid_part;      // [mid_items][kMidItemFloats] sums published by the medium-M GEMM (null: engine off)
  size_t mid_items;
  float* corr_lse;      // [Bmax] log-sum-exp of each sampling request's correction row
  float* corr_part;     // [Bmax][kCorrMaxSlices][4] per-slice winners of the correction draw
  uint32_t* corr_cnt;   // [Bmax] arrival counters of the correction slices (kept at zero between calls)
  int32_t* prefill_tok; // [Mrows] token ids of one batched-prefill forward
  int32_t* prefill_cnt; // [Bmax] prompt tokens to cache per request (batched prefill)
  int32_t* prefill_base; // [Bmax] each request's length when its batched prefill began
  size_t act_split;   // elements between splits of act_n / act_o
  size_t actf_split;  // elements between splits of act_f
  int Mmax;   // rows of a verify call (logits, LM-head statistics)
  int Mrows;  // rows of any forward (activations): Mmax, or more for prefill
  int NCmax, Rmax;
};

}  // namespace spade

struct spade_model_s {
  spade_config cfg;
  spade::Dims dims;
  spade::ArenaLayout lay;
  uint8_t* weights;
  uint8_t* work;
  spade::Workspace ws;
  int max_batch, max_gamma, max_len;
  int device;
  int n_cu;      // compute units of the device
  int gemm_wgs;  // persistent GEMM workgroups
  int wide_rt;   // 16-row tiles per workgroup of the wide-row GEMM: 0 chosen per launch, 1..3 fixed, -1 off
  int wide_p;    // panels per wave of the wide-row GEMM: 0 chosen per launch, 1..2 fixed
  int wide_ks;   // k-splits of its O and down projections: 0 chosen per launch, 1 off, 2 or 4 fixed
  int split_ks;  // k-splits of the split-K GEMM: 0 chosen per launch, 2 or 4 where it qualifies, -1 off
  int attn_merge;  // merge of one-chunk attention partials: 0 chosen per call, 1 last arrival, 2 second launch
  int attn_grouped;  // grouped-query chunks (one workgroup per K/V head and chunk): 0 where they apply, 1 off
  int corr_split;  // correction draws of sampling requests: 0/2 over vocabulary slices, 1 in the accept workgroup
  int prefill_rows;  // prompt rows per request of a prefill forward: 0 as many as the workspace holds, else at most this
  int big_gemm;  // large-M projection GEMM: 0 where it fills the chip, 1 off, 2 whenever more than 16 rows
  int mid_gemm;  // medium-M GEMM: 0 O, gate/up, down above mid_min_rows (to 144 rows), 1 off, 2 every projection of 17-144
  int mid_ks;    // its k-splits: 0 chosen per launch, 1..8 fixed
};

struct spade_kv_s {
  spade_model model;
  uint8_t* k;
  uint8_t* v;
  int32_t* lens;
  int32_t* pending;
  int max_batch, max_len;
  int stride;    // positions per (request, head) row of the cache: max_len rounded up to 32
  int* lens_ub;  // host upper bound of lens per request
  int last_rows; // rows (gamma + 1) of the last spade_verify on this cache: what a commit can add at most
  int last_B;    // requests of that call
  bool verified; // a spade_verify ran since the last commit or state change
  int* snap_ub;  // lens_ub at the last snapshot
};

namespace spade {

struct ForwardCall {
  int b0, nb, R;           // requests [b0, b0+nb), R rows each
  const int32_t* tokens;   // prefill: [R] ids; verify: NULL
  const int32_t* drafts;   // verify: [nb][R-1]
  bool want_logits;
  float* logits_out;       // [nb*R][V] (user buffer or workspace)
  const uint8_t* mode;     // verify: [nb] modes (LM-head statistics use 1/T on sampling rows)
  float inv_T;
  bool have_q;             // draft probabilities given
};

struct AcceptCall {
  int B, gamma, V;
  const float* logits;     // [B][gamma+1][V]
  const float* stats;      // [B*(gamma+1)][NU][3] from the LM head, or NULL
  int NU;
  int panels;              // > 0: stats is [B*(gamma+1)][panels][3], one entry per panel
  const int32_t* drafts;
  const float* q;
  const float* u;
  const uint8_t* mode;
  float inv_T;
  int32_t* n_out;
  int32_t* corr_out;
};

hipError_t launch_forward(spade_model m, spade_kv kv, const ForwardCall& fc, hipStream_t st);
// tiling of a wide-row launch: row tiles per workgroup, panels per wave, k-splits
struct WideChoice {
  int rt, p, ks;
};
WideChoice wide_choice(int kind, int M, int n_units, int NKB, int K, int n_cu, int fixed_rt, int fixed_p, int fixed_ks,
                       size_t cap_items, size_t cap_floats);
size_t wide_split_floats(int n_units, int M, int rt, int p);
int mid_k_splits(int n_units, int NKB, int n_cu, int fixed_ks);
int mid_min_rows(int kind);  // rows above which a projection kind runs on the medium-M GEMM by default
size_t mid_split_floats();  // published floats per panel group of a medium-M launch
int lm_stats_panels(spade_model m, int M);
hipError_t launch_softmax(const float* logits, int rows, int V, float invT, float* out, hipStream_t st);
hipError_t launch_prefill_batch(spade_model md, spade_kv kv, int B, const int32_t* tokens, int ld,
                                const int* n_cache, hipStream_t st);
hipError_t launch_prefill_one(spade_model md, spade_kv kv, int b, const int32_t* tokens, int n_cache,
                              hipStream_t st);
hipError_t launch_layer_gemm(spade_model m, spade_kv kv, int kind, int layer, const ForwardCall& fc,
                             hipStream_t st);
hipError_t launch_accept(spade_model m, const AcceptCall& ac, hipStream_t st);
// accept / correction with the library's static device scratch (no workspace)
hipError_t launch_accept_noalloc(const AcceptCall& ac, uint32_t* err, hipStream_t st);
size_t noalloc_scratch_bytes();
hipError_t launch_pack(spade_model m, int kind, int layer, const void* src, hipStream_t st);
hipError_t launch_commit(spade_kv kv, int B, int R, const int32_t* n, const int32_t* corr, hipStream_t st);
hipError_t launch_advance(spade_kv kv, int b, int count, const int32_t* pending_src, hipStream_t st);
hipError_t launch_copy_state(int B, int32_t* lens, int32_t* pending, const int32_t* src_lens,
                             const int32_t* src_pending, hipStream_t st);

}  // namespace spade
