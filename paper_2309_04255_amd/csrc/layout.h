// Packed-weight image and workspace layouts, shared by the host API and the
// kernels.  Everything here is plain integer arithmetic on the model shape.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "llmcad.h"

namespace llmcad {

constexpr int kNB = 16;          // output columns per n-block (one 16x16x32 MFMA)
constexpr int kStepK = 32;       // inputs per MFMA k-step
constexpr int kBlockBytes = kNB * kStepK * 2;  // one packed (n-block, k-step) block: 1 KiB
constexpr int kMaxNodes = LLMCAD_MAX_NODES;
constexpr int kAttnChunk = 128;     // key positions staged in LDS at once
constexpr int kAttnMaxSplits = 32;  // position splits per head
constexpr int kPassMaxGrid = 1024;  // workgroups of the pass
constexpr int kBarSlots = 16;       // grid-barrier counters
constexpr int kBarStride = 32;      // ints between barrier counters (128 bytes)

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
inline int round_up(int x, int a) { return (x + a - 1) / a * a; }
inline int cdiv(int x, int a) { return (x + a - 1) / a; }

// Rows a pass over n nodes computes: n rounded up to 16, 32, 48, 64 or 128
// (the row-block counts the kernels are built for).
inline int pass_rows(int n) {
  const int mb = cdiv(n, 16);
  return 16 * (mb <= 4 ? mb : 8);
}

struct Shape {
  int L, d, H, Dh, F, V;
  int Fp;     // F rounded up to 32 (SwiGLU width as stored; K of the down projection)
  int qkv_nb; // n-blocks of the QKV projection (3d / 16)
  int d_nb;   // n-blocks of the O and down projections (d / 16)
  int gu_nb;  // n-blocks of gate/up: each holds 8 gate and the matching 8 up columns (Fp / 8)
  int v_nb;   // n-blocks of the LM head (V / 16 rounded up)
  int ks_d, ks_f;  // k-steps over d and over Fp
  explicit Shape(const llmcad_config& c)
      : L(c.n_layers), d(c.d_model), H(c.n_heads), Dh(c.head_dim), F(c.d_ffn), V(c.vocab) {
    Fp = round_up(F, 32);
    qkv_nb = 3 * d / kNB;
    d_nb = d / kNB;
    gu_nb = Fp / 8;
    v_nb = cdiv(V, kNB);
    ks_d = d / kStepK;
    ks_f = Fp / kStepK;
  }
};

inline size_t packed_matrix_bytes(int nblocks, int ksteps) {
  return (size_t)nblocks * (size_t)ksteps * kBlockBytes;
}

// Byte offsets inside the packed image.
struct PackedLayout {
  size_t embed, final_norm, lm_head, globals_end;
  size_t layer_bytes;
  // offsets relative to the start of a layer
  size_t attn_norm, w_qkv, w_o, ffn_norm, w_gate_up, w_down;
  size_t total;
  explicit PackedLayout(const Shape& s) {
    size_t o = 0;
    embed = o;
    o = align_up(o + (size_t)s.V * s.d * 2, 4096);
    final_norm = o;
    o = align_up(o + (size_t)s.d * 2, 4096);
    lm_head = o;
    o = align_up(o + packed_matrix_bytes(s.v_nb, s.ks_d), 4096);
    globals_end = o;
    size_t p = 0;
    attn_norm = p;
    p = align_up(p + (size_t)s.d * 2, 4096);
    w_qkv = p;
    p = align_up(p + packed_matrix_bytes(s.qkv_nb, s.ks_d), 4096);
    w_o = p;
    p = align_up(p + packed_matrix_bytes(s.d_nb, s.ks_d), 4096);
    ffn_norm = p;
    p = align_up(p + (size_t)s.d * 2, 4096);
    w_gate_up = p;
    p = align_up(p + packed_matrix_bytes(s.gu_nb, s.ks_d), 4096);
    w_down = p;
    p = align_up(p + packed_matrix_bytes(s.d_nb, s.ks_f), 4096);
    layer_bytes = p;
    total = globals_end + (size_t)s.L * layer_bytes;
  }
  size_t layer(int l) const { return globals_end + (size_t)l * layer_bytes; }
};

// Byte offsets inside a workspace sized for passes of up to max_n nodes
// (row count Mp = pass_rows(max_n)).
// Buffers handed from one phase of a pass to the next are written once per
// pass (one copy per layer), so no cache can hold a stale copy of them.
struct WorkspaceLayout {
  int Mp;
  int n_tile_counters, n_head_counters;
  size_t counters;     // int32: tiles [n_tile] | heads [H] | lm | exit | status | spare
  size_t counters_bytes;
  size_t bar;          // int32 [kBarSlots][kBarStride] grid-barrier counters
  size_t scratch_out;  // int32 [128 + 2] path/len/next sink for prefill
  size_t tree;         // int32 tok[128] | parent[128] | depth[128] | pos[128] | uint32 anc[128][4]
  size_t trace;        // int64 [8][2 + 5L][6]    phase timestamps (diagnostics)
  size_t amax;         // int32 [Mp]              per-node greedy token
  size_t lm_val;       // fp32 [G + v_nb][Mp]     argmax partials (value)
  size_t lm_idx;       // int32 [G + v_nb][Mp]    argmax partials (column)
  size_t xs;           // fp32 [2L+1][Mp][d]      residual stream versions
  size_t ssqs;         // fp32 [2L+1][d/16][Mp]   their per-n-block sums of squares
  size_t qs;           // bf16 [L][Mp][d]         queries after the rotary embedding
  size_t os;           // bf16 [L][Mp][d]         attention output
  size_t hs;           // bf16 [L][Mp][Fp]        SwiGLU product
  size_t part;         // fp32 [kPassMaxGrid][2][Mp][16] stream-K partial n-blocks
  size_t attn_o;       // fp32 [H][S][Mp][Dh]     per-split unnormalised outputs
  size_t attn_ml;      // fp32 [H][S][Mp][2]      per-split running max and sum
  size_t total;
  WorkspaceLayout(const Shape& s, int max_n) {
    Mp = pass_rows(max_n);
    size_t o_ = 0;
    auto take = [&](size_t bytes) {
      size_t at = o_;
      o_ = align_up(o_ + bytes, 256);
      return at;
    };
    // Fixed-size buffers first: their offsets do not depend on the node count.
    int tiles = s.v_nb;
    if (s.qkv_nb > tiles) tiles = s.qkv_nb;
    if (s.gu_nb > tiles) tiles = s.gu_nb;
    if (s.d_nb > tiles) tiles = s.d_nb;
    n_tile_counters = tiles;
    n_head_counters = s.H;
    counters_bytes = (size_t)(n_tile_counters + n_head_counters + 4) * 4;
    counters = take(counters_bytes);
    bar = take((size_t)kBarSlots * kBarStride * 4);
    scratch_out = take((128 + 2) * 4);
    tree = take(4 * 128 * 4 + 128 * 4 * 4);
    trace = take((size_t)8 * (2 + 5 * s.L) * 6 * 8);
    amax = take((size_t)Mp * 4);
    lm_val = take((size_t)(kPassMaxGrid + s.v_nb) * Mp * 4);
    lm_idx = take((size_t)(kPassMaxGrid + s.v_nb) * Mp * 4);
    xs = take((size_t)(2 * s.L + 1) * Mp * s.d * 4);
    ssqs = take((size_t)(2 * s.L + 1) * s.d_nb * Mp * 4);
    qs = take((size_t)s.L * Mp * s.d * 2);
    os = take((size_t)s.L * Mp * s.d * 2);
    hs = take((size_t)s.L * Mp * s.Fp * 2);
    part = take((size_t)kPassMaxGrid * 2 * Mp * kNB * 4);
    attn_o = take((size_t)s.H * kAttnMaxSplits * Mp * s.Dh * 4);
    attn_ml = take((size_t)s.H * kAttnMaxSplits * Mp * 2 * 4);
    total = o_;
  }
  size_t lm_cnt() const { return counters + (size_t)(n_tile_counters + n_head_counters) * 4; }
  size_t exit_cnt() const { return lm_cnt() + 4; }
  size_t status() const { return lm_cnt() + 8; }
};

}  // namespace llmcad
