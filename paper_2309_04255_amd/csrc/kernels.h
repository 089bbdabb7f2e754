// Launchers of the library's kernels (host side).  Each returns the HIP status
// of its launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device.h"

namespace llmcad {

// ---- weight packing (pack.hip)
enum PackKind { PACK_PLAIN = 0, PACK_QKV_ROPE = 1, PACK_GATE_UP = 2 };
hipError_t launch_pack(const void* w, int N, int K, void* out, int tiles, int ksteps, int kind,
                       int H, int Dh, int F, hipStream_t st);

// ---- tree preparation + embedding (tree.hip)
struct TreeArgs {
  int32_t tok[128];
  int32_t parent[128];
};
hipError_t launch_embed(const TreeArgs& tree, int n, int Mp, int d, int prefix_len,
                        const void* tok_embed, void* ws_tree, float* x, float* ssq,
                        hipStream_t st);

// ---- skinny GEMM with fused prologue/epilogue (gemm.hip)
enum Prologue { PRO_BF16 = 0, PRO_NORM = 1 };
enum Epilogue { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_LOGITS = 3 };

struct GemmParams {
  const void* w;  // packed matrix
  int ksteps;     // k-steps of 32 per tile
  int tiles;      // 64-column tiles
  int ksplit;     // k-splits per tile
  int n;          // valid rows
  int Mp;         // padded rows (multiple of 16)
  // A operand
  const void* a;  // PRO_BF16: bf16 [Mp][lda]
  int lda;
  const float* x;    // PRO_NORM: fp32 [Mp][d]
  const float* ssq;  // PRO_NORM: fp32 [ssq_tiles][Mp]
  int ssq_tiles;
  const void* gain;  // PRO_NORM: bf16 [d]
  float eps;
  float inv_d;
  int d;  // row length of x
  // split-K
  float* part;    // fp32 [tiles * ksplit][Mp][64]
  int* counters;  // int32 [tiles], zero on entry, left zero
  // EPI_QKV
  void* q_out;    // bf16 [Mp][d]
  void* k_cache;  // bf16 [H][cap][Dh] of this layer
  void* v_cache;
  int cap, prefix_len, H, Dh;
  const int* pos;  // int32 [n]
  float log2_theta;
  // EPI_RESID
  float* x_out;    // fp32 [Mp][d]
  float* ssq_out;  // fp32 [tiles][Mp]
  // EPI_SWIGLU
  void* h_out;  // bf16 [Mp][ldh]
  int ldh;
  // EPI_LOGITS
  float* logits;  // fp32 [n - row_lo][V] or null
  int V;
  int row_lo;
  float* lm_val;  // fp32 [tiles][Mp]
  int* lm_idx;    // int32 [tiles][Mp]
  int* lm_counter;
  int* amax;       // int32 [Mp]
  const int* tree_tok;
  const int* tree_parent;
  const int* tree_depth;
  int* path;
  int* accept_len;
  int* next_token;
};
hipError_t launch_gemm(int pro, int epi, int mb, const GemmParams& p, hipStream_t st);

// ---- tree-masked attention (attention.hip)
struct AttnParams {
  const void* q;        // bf16 [Mp][H*Dh] rotated queries
  const void* k_cache;  // bf16 [H][cap][Dh] of this layer
  const void* v_cache;
  void* o_out;          // bf16 [Mp][H*Dh]
  float* part_o;        // fp32 [H][S][Mp][Dh]
  float* part_ml;       // fp32 [H][S][Mp][2]
  int* counters;        // int32 [H]
  const uint32_t* anc;  // uint32 [128][4] ancestor-or-self bit sets
  int n, Mp, H, Dh, cap, prefix_len;
  int splits;   // position splits per head
  int nchunks;  // 64-wide key chunks covering [0, prefix_len + n)
  float scale_log2;  // log2(e) / sqrt(Dh)
};
hipError_t launch_attention(int mb, const AttnParams& p, hipStream_t st);

// ---- persistent single-launch pass (pass.hip)
struct PassParams {  // see pass.hip for the phase structure
  int L, d, H, Dh, F, Fp, V;
  float eps, inv_d, log2_theta, scale_log2;
  int n, Mp, prefix_len, cap, G;
  const char* packed;
  long long o_embed, o_final_norm, o_lm, layer0, layer_bytes;
  long long o_attn_norm, o_qkv, o_o, o_ffn_norm, o_gu, o_down;
  int ks_d, ks_f, qkv_tiles, d_tiles, gu_tiles, v_tiles;
  bf16* k_cache;
  bf16* v_cache;
  int* tree;
  float* x;    // [2L+1][Mp][d]
  float* ssq;  // [2L+1][d_tiles][Mp]
  bf16* q;     // [L][Mp][d]
  bf16* o;     // [L][Mp][d]
  bf16* h;     // [L][Mp][Fp]
  float* part; // [G][2][Mp][64]
  float* attn_o;
  float* attn_ml;
  int attn_splits;
  int* tile_cnt;
  int* head_cnt;
  int* lm_cnt;
  int* bar;
  int* exit_cnt;
  int* status;
  float* lm_val;
  int* lm_idx;
  int* amax;
  float* logits;
  int row_lo;
  int* path;
  int* accept_len;
  int* next_token;
  int spin_limit;
  long long* trace;  // diagnostics: [8][2 + 5L][3] phase timestamps, or null
};
hipError_t launch_pass(int mb, const PassParams& p, const TreeArgs& tree, hipStream_t st);
int pass_occupancy(int mb, int dh);  // resident workgroups per CU (0 if unavailable)

}  // namespace llmcad
