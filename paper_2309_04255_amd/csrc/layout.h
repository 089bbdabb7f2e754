// Packed-weight image and workspace layouts, shared by the host API and the
// kernels.  Everything here is plain integer arithmetic on the model shape.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "llmcad.h"

namespace llmcad {

constexpr int kTileN = 64;       // output columns per GEMM tile (4 MFMA n-blocks of 16)
constexpr int kStepK = 32;       // inputs per MFMA k-step (16x16x32 bf16)
constexpr int kBlockBytes = kTileN * kStepK * 2;  // one packed (tile, k-step) block: 4 KiB
constexpr int kMaxNodes = LLMCAD_MAX_NODES;
constexpr int kAttnChunk = 64;   // key positions staged in LDS per attention step
constexpr int kGemmMaxWgs = 4096;   // bound on (tiles x k-splits) of one GEMM launch
constexpr int kAttnMaxWgs = 1024;   // bound on (heads x position splits)

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
inline int round_up(int x, int a) { return (x + a - 1) / a * a; }
inline int cdiv(int x, int a) { return (x + a - 1) / a; }

struct Shape {
  int L, d, H, Dh, F, V;
  int Fp;       // F rounded up to 32 (SwiGLU width as stored)
  int Vp;       // V rounded up to 64
  int d_tiles;  // d / 64
  int v_tiles;  // Vp / 64
  int qkv_tiles, gu_tiles;
  int ks_d, ks_f;  // k-steps over d and over Fp
  explicit Shape(const llmcad_config& c)
      : L(c.n_layers), d(c.d_model), H(c.n_heads), Dh(c.head_dim), F(c.d_ffn), V(c.vocab) {
    Fp = round_up(F, 32);
    Vp = round_up(V, 64);
    d_tiles = d / 64;
    v_tiles = Vp / 64;
    qkv_tiles = 3 * d / 64;
    gu_tiles = Fp / 32;
    ks_d = d / 32;
    ks_f = Fp / 32;
  }
};

inline size_t packed_matrix_bytes(int tiles, int ksteps) {
  return (size_t)tiles * (size_t)ksteps * kBlockBytes;
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
    o = align_up(o + packed_matrix_bytes(s.v_tiles, s.ks_d), 4096);
    globals_end = o;
    size_t p = 0;
    attn_norm = p;
    p = align_up(p + (size_t)s.d * 2, 4096);
    w_qkv = p;
    p = align_up(p + packed_matrix_bytes(s.qkv_tiles, s.ks_d), 4096);
    w_o = p;
    p = align_up(p + packed_matrix_bytes(s.d_tiles, s.ks_d), 4096);
    ffn_norm = p;
    p = align_up(p + (size_t)s.d * 2, 4096);
    w_gate_up = p;
    p = align_up(p + packed_matrix_bytes(s.gu_tiles, s.ks_d), 4096);
    w_down = p;
    p = align_up(p + packed_matrix_bytes(s.d_tiles, s.ks_f), 4096);
    layer_bytes = p;
    total = globals_end + (size_t)s.L * layer_bytes;
  }
  size_t layer(int l) const { return globals_end + (size_t)l * layer_bytes; }
};

// Split of an attention pass over key positions: every head's positions
// [0, P + n) are cut into 64-wide chunks, and each workgroup takes a
// contiguous run of chunks.
constexpr int kAttnMaxSplits = 32;  // position splits per head
constexpr int kPassMaxGrid = 1024;  // workgroups of the persistent pass
inline int attn_max_splits(int H) {
  int s = kAttnMaxWgs / H;
  if (s > kAttnMaxSplits) s = kAttnMaxSplits;
  return s < 1 ? 1 : s;
}

// Byte offsets inside a workspace sized for max_n nodes.
struct WorkspaceLayout {
  int Mp;
  size_t tree;       // int32 tok[128], parent[128], depth[128], pos[128]; uint32 anc[128][4]
  size_t x;          // fp32 [Mp][d]       residual stream
  size_t ssq;        // fp32 [d/64][Mp]    per-tile sums of squares of x
  size_t q;          // bf16 [Mp][d]       rotated queries
  size_t o;          // bf16 [Mp][d]       attention output
  size_t h;          // bf16 [Mp][Fp]      SwiGLU product
  size_t amax;       // int32 [Mp]         per-node greedy token
  size_t lm_val;     // fp32 [Vt][Mp]      per-tile row maxima of the logits
  size_t lm_idx;     // int32 [Vt][Mp]     their columns
  size_t gemm_part;  // fp32 [kGemmMaxWgs][Mp][64] split-K partial tiles
  size_t attn_o;     // fp32 [H][S][Mp][Dh] per-split unnormalised outputs
  size_t attn_ml;    // fp32 [H][S][Mp][2]  per-split running max and sum
  size_t scratch_out;  // int32 [128 + 2]  path/len/next sink for prefill
  // persistent pass: one buffer per producing phase (written once per pass)
  size_t xs;         // fp32 [2L+1][Mp][d]        residual stream versions
  size_t ssqs;       // fp32 [2L+1][d/64][Mp]     their per-tile sums of squares
  size_t qs;         // bf16 [L][Mp][d]
  size_t os;         // bf16 [L][Mp][d]
  size_t hs;         // bf16 [L][Mp][Fp]
  size_t part_sk;    // fp32 [kPassMaxGrid][2][Mp][64] stream-K partial tiles
  size_t trace;      // int64 [8][2 + 5L][6] phase timestamps (diagnostics)
  size_t bar;        // int32 [16][32] grid-barrier slots, one per 128-byte line
  size_t counters;   // int32 [ncounters]: gemm tiles | heads | lm | barrier | exit | status
  int n_gemm_counters, n_attn_counters;
  size_t counters_bytes;
  size_t total;
  WorkspaceLayout(const Shape& s, int max_n) {
    Mp = round_up(max_n, 16);
    const int S = attn_max_splits(s.H);
    size_t o_ = 0;
    auto take = [&](size_t bytes) {
      size_t at = o_;
      o_ = align_up(o_ + bytes, 256);
      return at;
    };
    // Counters and small fixed-size buffers first, so their offsets do not
    // depend on the pass's node count.
    int max_tiles = s.v_tiles;
    if (s.qkv_tiles > max_tiles) max_tiles = s.qkv_tiles;
    if (s.gu_tiles > max_tiles) max_tiles = s.gu_tiles;
    n_gemm_counters = max_tiles;
    n_attn_counters = s.H;
    counters_bytes = (size_t)(n_gemm_counters + n_attn_counters + 4) * 4;
    counters = take(counters_bytes);
    bar = take(16 * 32 * 4);
    scratch_out = take((128 + 2) * 4);
    tree = take(4 * 128 * 4 + 128 * 4 * 4);
    x = take((size_t)Mp * s.d * 4);
    ssq = take((size_t)s.d_tiles * Mp * 4);
    q = take((size_t)Mp * s.d * 2);
    o = take((size_t)Mp * s.d * 2);
    h = take((size_t)Mp * s.Fp * 2);
    amax = take((size_t)Mp * 4);
    lm_val = take((size_t)s.v_tiles * Mp * 4);
    lm_idx = take((size_t)s.v_tiles * Mp * 4);
    gemm_part = take((size_t)kGemmMaxWgs * Mp * 64 * 4);
    attn_o = take((size_t)s.H * S * Mp * s.Dh * 4);
    attn_ml = take((size_t)s.H * S * Mp * 2 * 4);
    xs = take((size_t)(2 * s.L + 1) * Mp * s.d * 4);
    ssqs = take((size_t)(2 * s.L + 1) * s.d_tiles * Mp * 4);
    qs = take((size_t)s.L * Mp * s.d * 2);
    os = take((size_t)s.L * Mp * s.d * 2);
    hs = take((size_t)s.L * Mp * s.Fp * 2);
    part_sk = take((size_t)kPassMaxGrid * 2 * Mp * 64 * 4);
    trace = take((size_t)8 * (2 + 5 * s.L) * 6 * 8);
    total = o_;
  }
};

}  // namespace llmcad
