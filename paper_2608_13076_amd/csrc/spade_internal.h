// Internal declarations shared by the C ABI (api.cpp) and the kernels
// (kernels.hip).  Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/spade.h"

namespace spade {

constexpr int kPanel = 16;          // weight rows per MFMA tile (one panel)
constexpr int kTileBytes = 8192;    // one panel x one k-block, in the arena
constexpr int kMaxRowsPerGemm = 32; // rows handled by one GEMM launch
constexpr int kPrefillRows = 16;    // tokens per prefill forward
constexpr int kMaxR = 16;           // rows per request in one forward (gamma <= 15)
constexpr int kAttnChunkMin = 64;

enum GemmKind { GEMM_QKV = 0, GEMM_O = 1, GEMM_GU = 2, GEMM_DOWN = 3, GEMM_LM = 4 };

inline int kblock_of(int weight_dtype) { return weight_dtype == SPADE_BF16 ? 256 : 128; }
inline int panels_per_unit(int kind) { return (kind == GEMM_QKV || kind == GEMM_GU) ? 2 : 1; }

// Weight panel (16 rows of the logical [N, K] matrix) held by panel slot pp of
// unit u.  The arena stores units in order; within a unit, k-block major and
// panel minor, so the k-range a wave streams is one contiguous block.
//   QKV: N = 3d.  Unit u covers section s (q, k, v), head h and panel w of the
//        first half of the head; its partner panel holds features + hd/2, so
//        the RoPE pair (i, i + hd/2) lands in the same thread.
//   GU:  N = 2F (gate rows, then up rows).  Unit u = gate panel u + up panel u.
//   others: unit u = panel u.
__host__ __device__ inline int unit_panel(int kind, int u, int pp, int d_model, int head_dim, int d_ffn) {
  if (kind == GEMM_QKV) {
    const int upsec = d_model / 32, uph = head_dim / 32;
    const int s = u / upsec, rem = u % upsec;
    const int h = rem / uph, w = rem % uph;
    return s * (d_model / 16) + h * (head_dim / 16) + w + pp * uph;
  }
  if (kind == GEMM_GU) return u + pp * (d_ffn / 16);
  return u;
}

struct Dims {
  int L, d, H, hd, F, V, Vpad, wdt, kvdt;
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
  float* x;          // [Mmax][d] residual stream
  void* act_n;       // normed GEMM input, split bf16 [S][Mmax][d] or f32 [Mmax][d]
  void* act_o;       // attention output (O-projection input)
  void* act_f;       // SwiGLU output (down-projection input) [S][Mmax][F]
  float* ssq;        // [Mmax][d/16] sum-of-squares partials of x
  float* q;          // [Mmax][d] rotated queries
  float* attn_o;     // [Bmax][H][NCmax][Rmax][hd] chunk partial outputs
  float* attn_ml;    // [Bmax][H][NCmax][Rmax][2] chunk max / sum
  uint32_t* attn_cnt;// [Bmax][H] arrival counters (kept at zero between calls)
  float* logits;     // [Mmax][V]
  float* stats;      // [Mmax][NU][3] LM-head per-unit max / sumexp / argmax
  float* rope;       // [max_len][hd/2][2] cos, sin
  float* inv_temp;   // [Bmax]
  int32_t* tokens;   // [Mmax] staging for prefill tokens
  uint32_t* err;     // device error word
  size_t act_split;  // elements between splits of act_n / act_o
  size_t actf_split; // elements between splits of act_f
  int Mmax, NCmax, Rmax;
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
  int S;  // activation splits for bf16 GEMMs
  int device;
};

struct spade_kv_s {
  spade_model model;
  uint8_t* k;
  uint8_t* v;
  int32_t* lens;
  int32_t* pending;
  int max_batch, max_len;
  int* lens_ub;  // host upper bound of lens per request
};

namespace spade {

// Launchers (kernels.hip).  All return hipError_t of the launch.
struct ForwardCall {
  int b0, nb, R;                  // requests [b0, b0+nb), R rows each
  const int32_t* tokens;          // prefill: [R] ids; verify: NULL
  const int32_t* drafts;          // verify: [nb][R-1]
  bool want_logits;
  float* logits_out;              // [nb*R][V] (user buffer or workspace)
};

hipError_t launch_forward(spade_model m, spade_kv kv, const ForwardCall& fc, hipStream_t st);
hipError_t launch_accept(spade_model m, int B, int gamma, int V, const float* logits, bool have_stats,
                         const int32_t* drafts, const float* q, const float* u, const uint8_t* mode,
                         float temperature, int32_t* n_out, int32_t* corr_out, hipStream_t st);
hipError_t launch_pack(spade_model m, int kind, int layer, const void* src, hipStream_t st);
hipError_t launch_commit(spade_kv kv, int B, const int32_t* n, const int32_t* corr, hipStream_t st);
hipError_t launch_advance(spade_kv kv, int b, int count, const int32_t* pending_src, hipStream_t st);
hipError_t launch_set_inv_temp(spade_model m, int B, const uint8_t* mode, float temperature,
                               bool have_q, hipStream_t st);

}  // namespace spade
