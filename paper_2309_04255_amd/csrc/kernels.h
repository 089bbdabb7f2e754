// Launchers of the library's kernels (host side).  Each returns the HIP status
// of its launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device.h"
#include "layout.h"

namespace llmcad {

// ---- weight packing (pack.hip)
// aux: F (the FFN width) for PACK_GATE_UP, the head dimension for
// PACK_QKV_ROPE, unused for PACK_PLAIN.
enum PackKind { PACK_PLAIN = 0, PACK_GATE_UP = 1, PACK_QKV_ROPE = 2 };
hipError_t launch_pack(const void* w, int N, int K, void* out, int nblocks, int ksteps, int kind,
                       int aux, hipStream_t st);
// 4-bit matrix: codes uint8 [N][K/2] and bf16 scales [N][K/128] -> packed
// codes [nblocks][groups] x 1 KiB and packed scales [nblocks][groups][16].
hipError_t launch_pack_q4(const void* codes, const void* scales, int N, int K, void* out_codes, void* out_scales,
                          int nblocks, int groups, int kind, int aux, hipStream_t st);

// ---- rollback to the verified sequence (commit.hip): for each of the
// layers_heads (layer, head) row sets of the cache, slot prefix_len + path[k]
// -> prefix_len + k for k = 1..*accept_len (path and accept_len in device
// memory; n = the pass's node count bounds both).  LDS: 2 n dh bf16.
hipError_t launch_commit(void* k_cache, void* v_cache, int layers_heads, int cap, int prefix_len, const int* path,
                         const int* accept_len, int n, int dh, hipStream_t st);

// ---- the verification pass as one persistent launch (pass.hip)
struct TreeArgs {
  int32_t tok[128];
  int32_t parent[128];
};

// Set in PassParams::magic by the host; the kernel checks it where it reads
// the parameters in place.
constexpr int kPassMagic = 0x4c4d4342;

// One GEMM step's shape and where its weights live.
struct StepPlan {
  int nblocks, ksteps;  // 16-column blocks; 32-input k-steps (4-bit: 128-input scale groups)
  long long w_off;      // packed matrix (4-bit: its codes): offset from the packed image (globals) or the layer start
  long long s_off;      // 4-bit: the packed scales, offset as w_off
  int layer_rel;        // 1 if w_off is relative to the layer's start
  int q4;               // 1: 4-bit codes with group scales
  int split;            // split-K: workgroups sharing each group of column blocks (1: none; 2 or 4)
  int wl_cap;           // weight stages per wave copied to LDS before the step's barrier, at most
  int wide;             // 16- and 32-row passes: tiles of up to 9 blocks instead of 8
};

// Must stay the first kernel argument of the pass kernel.
struct PassParams {
  int magic;
  // model
  int L, d, H, Dh, F, Fp, V;
  float eps, inv_d, log2_theta, scale_log2;
  // pass: rows n = nodes [m0, nt) of a tree of nt nodes (m0 = 0: all of it);
  // nodes [0, m0) were computed by earlier passes, their K/V are in slots
  // prefix_len + i
  int n, Mp, prefix_len, cap, G;
  int m0, nt;
  // packed weights
  const char* packed;
  long long o_embed, o_final_norm, layer0, layer_bytes;
  long long o_attn_norm, o_ffn_norm;
  int d_nb;
  StepPlan step[kSteps];
  // KV cache: K [L][H][cap][Dh], V transposed per head [L][H][Dh][cap]
  bf16* k_cache;
  bf16* v_cache;
  // workspace
  int* tree;        // tok | parent | depth | pos | anc
  const char* zero; // kZeroBytes of zeros
  float* rope;      // [Mp][Dh/2][2] cos, sin of every node's rotary angles
  float* x;         // [2L+1][Mp][d]
  bf16* xg;         // [2L+1] x fragment-order [Mp][d]: bf16(x * g), g the gain of the norm that reads x
  bf16* xnf;        // fragment-order [Mp][d]: the final norm's output bf16(x rstd g), the LM head's input
  float* ssq;       // [2L+1][d/16][Mp]
  int ssq_regs;     // 1 if a norm step's tiles hold its sums of squares in registers
                    // (Mp <= 32 and at most 8 blocks per chunk of d/16 / (1024 / Mp) blocks)
  bf16* q;          // [L][Mp][d]   queries after the rotary embedding
  bf16* o;          // [L] x fragment-order [Mp][d]
  bf16* h;          // [L] x fragment-order [Mp][Fp]
  int* lm_cnt;
  int* exit_cnt;
  int* status;
  int* bar;         // [kBarSlots][kBarStride]
  float* attn_o;    // [H][MB][KS][16][Dh] key-split partial outputs (unnormalised)
  float* attn_ml;   // [H][MB][KS][16][2]  their running max and sum
  int attn_splits;  // KS, key splits per (head, row block): 1 to 4 (the split's 32-key steps contiguous)
  int* head_cnt;    // [H][MB] arrivals of the key splits
  float* part;      // split-K partial tiles: per workgroup w, [cdiv(blocks, G/S)][MB] x 1 KiB
                    // (fp32 [64 lanes][4]) from slot w cdiv(blocks, G/S)
  int* grp_cnt;     // [O, down][kPassMaxGrid / 2] arrivals of the workgroups of each split-K group
  float* lm_val;    // [Mp][G] LM-head argmax per row and workgroup
  int* lm_idx;
  float* lm_sum;    // [Mp][G] sum of exp(logit - the workgroup's max) over its columns (with cand)
  // candidate summaries (llmcad_extend_tree_candidates): per computed row the
  // argmax, softmax normaliser and every token above cand_thr, or null
  llmcad_candidates* cand;
  float cand_thr;
  int* amax;        // [Mp]
  // outputs
  float* logits;    // rows [row_lo, n) x V, or null
  int row_lo;
  int* path;
  int* accept_len;
  int* next_token;
  // control
  int spin_limit;    // bound of every wait loop (polls)
  int attn_prefetch; // 1: the attention fetches its prefix steps before its barrier (0: all after)
  int row_tiles;     // 1: GEMM phases of passes of 64+ rows take row-split tiles (waves split rows)
  long long* trace;  // diagnostics: [G][4 + 5L][8] phase timestamps, or null
};

// mb16: 16-row blocks of the pass (Mp / 16: 1, 2, 4 or 8).
hipError_t launch_pass(int mb16, const PassParams& p, const TreeArgs& tree, hipStream_t st);
int pass_occupancy(int mb16, int dh, bool wide);  // resident workgroups per CU (0 if unavailable)
size_t pass_lds_bytes(int mb16, int dh);


}  // namespace llmcad
