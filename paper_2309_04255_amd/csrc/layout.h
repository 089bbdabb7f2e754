// Packed-weight image, GEMM work plans and workspace layout, shared by the
// host API and the kernels.  Everything here is plain integer arithmetic on
// the model shape.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "llmcad.h"

namespace llmcad {

// One packed weight block feeds one 16x16x32 MFMA: 16 output columns x 32
// inputs, bf16, 1 KiB.
constexpr int kNB = 16;                        // output columns per block
constexpr int kStepK = 32;                     // inputs per k-step
constexpr int kBlockBytes = kNB * kStepK * 2;  // 1 KiB
// Group-quantised 4-bit weights: one scale per output column and group of
// kQ4Group inputs; a packed group of one 16-column block is 1 KiB of codes
// (16 columns x 128 inputs x 4 bits) plus its 16 bf16 scales.
constexpr int kQ4Group = 128;
constexpr int kQ4BlockBytes = kNB * kQ4Group / 2;  // 1 KiB
constexpr int kQ4ScaleBytes = kNB * 2;
constexpr int kMaxNodes = LLMCAD_MAX_NODES;
constexpr int kAttnMaxSplits = 4;   // key splits per (head, 16-row block)
constexpr int kMaxSplitK = 4;       // workgroups sharing the k-steps of a group of column blocks
constexpr int kPassMaxGrid = 1024;  // workgroups of the pass
constexpr int kBarSlots = 16;       // grid-barrier counters
constexpr int kBarStride = 32;      // ints between barrier counters (128 bytes)
constexpr int kZeroBytes = 4096;    // zeros (padding reads)

// Phases of a pass: tree prep + embedding, a barrier that publishes the
// rotary table, five per layer, the final norm, and the LM head.
#if defined(__HIPCC__)
__host__ __device__
#endif
inline int pass_phases(int L) { return 4 + 5 * L; }

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
inline int round_up(int x, int a) { return (x + a - 1) / a * a; }
inline int cdiv(int x, int a) { return (x + a - 1) / a; }

// Rows a pass over n nodes computes: n rounded up to 16, 32, 64 or 128 (one,
// two, four or eight 16-row MFMA blocks).
inline int pass_rows(int n) {
  const int mb = cdiv(n, 16);
  return 16 * (mb <= 1 ? 1 : mb <= 2 ? 2 : mb <= 4 ? 4 : 8);
}

struct Shape {
  int L, d, H, Dh, F, V;
  bool q4;     // layer matrices group-quantised to 4 bits (embedding, LM head and norms bf16)
  int Fp;      // F rounded up to 32 (SwiGLU width as stored; K of the down projection)
  int qkv_nb;  // column blocks of the QKV projection (3d / 16)
  int d_nb;    // column blocks of the O and down projections (d / 16)
  int gu_nb;   // column blocks of gate/up: each holds 8 gate and the matching 8 up columns (Fp / 8)
  int v_nb;    // column blocks of the LM head (V / 16 rounded up)
  int ks_d, ks_f;  // k-steps over d and over Fp
  int gs_d, gs_f;  // 4-bit weights: scale groups over d and over Fp
  explicit Shape(const llmcad_config& c)
      : L(c.n_layers), d(c.d_model), H(c.n_heads), Dh(c.head_dim), F(c.d_ffn), V(c.vocab),
        q4(c.weight_bits == 4) {
    Fp = round_up(F, kStepK);
    gs_d = d / kQ4Group;
    gs_f = Fp / kQ4Group;
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
// A 4-bit matrix: codes [nblocks][groups] x 1 KiB, then scales [nblocks][groups][16] bf16.
inline size_t q4_codes_bytes(int nblocks, int groups) { return (size_t)nblocks * groups * kQ4BlockBytes; }
inline size_t q4_matrix_bytes(int nblocks, int groups) {
  return q4_codes_bytes(nblocks, groups) + (size_t)nblocks * groups * kQ4ScaleBytes;
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
    // a layer matrix of nb blocks over K = 32 ks inputs, bf16 or 4-bit
    auto mat = [&](int nb, int ks, int gs) { return s.q4 ? q4_matrix_bytes(nb, gs) : packed_matrix_bytes(nb, ks); };
    size_t p = 0;
    attn_norm = p;
    p = align_up(p + (size_t)s.d * 2, 4096);
    w_qkv = p;
    p = align_up(p + mat(s.qkv_nb, s.ks_d, s.gs_d), 4096);
    w_o = p;
    p = align_up(p + mat(s.d_nb, s.ks_d, s.gs_d), 4096);
    ffn_norm = p;
    p = align_up(p + (size_t)s.d * 2, 4096);
    w_gate_up = p;
    p = align_up(p + mat(s.gu_nb, s.ks_d, s.gs_d), 4096);
    w_down = p;
    p = align_up(p + mat(s.d_nb, s.ks_f, s.gs_f), 4096);
    layer_bytes = p;
    total = globals_end + (size_t)s.L * layer_bytes;
  }
  size_t layer(int l) const { return globals_end + (size_t)l * layer_bytes; }
};

// The GEMM steps of a pass.
enum Step { STEP_QKV = 0, STEP_O = 1, STEP_GATE_UP = 2, STEP_DOWN = 3, STEP_LM = 4, kSteps = 5 };

// Column blocks of each step.  A step's blocks are dealt out in contiguous
// runs: workgroup w of G takes blocks [w nb / G, (w + 1) nb / G), over the
// full K, in tiles of a few blocks each.
inline int step_blocks(const Shape& s, int step) {
  switch (step) {
    case STEP_QKV: return s.qkv_nb;
    case STEP_O: return s.d_nb;
    case STEP_GATE_UP: return s.gu_nb;
    case STEP_DOWN: return s.d_nb;
    default: return s.v_nb;
  }
}
inline int step_ksteps(const Shape& s, int step) { return step == STEP_DOWN ? s.ks_f : s.ks_d; }
// 4-bit layer steps: scale groups over K (the LM head stays bf16)
inline int step_groups(const Shape& s, int step) { return step == STEP_DOWN ? s.gs_f : s.gs_d; }

// Byte offsets inside a workspace sized for passes of up to max_n nodes on
// a device with G workgroups (row count Mp = pass_rows(max_n)).  Buffers
// handed from one phase of a pass to the next are written once per pass (one
// copy per layer), so no cache can hold a stale copy of them; buffers reused
// within a pass (attention partials, counters) are accessed with
// device-coherent operations only.
//
// Fragment order (xg, o, h): a bf16 [Mp][K] matrix stored as 1 KiB blocks,
// block (k-step s, row block rb) at ((s Mp/16 + rb) KiB), lane l's 16 bytes
// = row 16 rb + l % 16, inputs 32 s + 8 (l / 16) .. + 7: the A operand of
// one 16x16x32 MFMA, loaded with one contiguous 1 KiB read.
struct WorkspaceLayout {
  int Mp;
  int n_head_counters;
  int n_group_counters;
  size_t part_slots;   // 1 KiB x Mp/16 partial tiles the split-K region holds
  size_t counters;     // int32: (head, row block) [H][8] | lm | exit | status | split-K groups
  size_t counters_bytes;
  size_t bar;          // int32 [kBarSlots][kBarStride] grid-barrier counters
  size_t zero;         // kZeroBytes of zeros (never written by a pass)
  size_t scratch_out;  // int32 [128 + 2] path/len/next sink for prefill
  size_t tree;         // int32 tok[128] | parent[128] | depth[128] | pos[128] | uint32 anc[128][4]
  size_t rope;         // fp32 [Mp][Dh/2][2]      cos, sin of every node's rotary angles
  size_t amax;         // int32 [Mp]              per-node greedy token
  size_t lm_val;       // fp32 [Mp][G]            LM-head argmax per row and workgroup
  size_t lm_idx;       // int32 [Mp][G]
  size_t lm_sum;       // fp32 [Mp][G]            its softmax normaliser (candidate summaries)
  size_t xs;           // fp32 [2L+1][Mp][d]      residual stream versions
  size_t xgs;          // bf16 [2L+1] x (Mp x d, fragment order)  bf16(x * g) (g: its norm's gain)
  size_t xnf;          // bf16 Mp x d, fragment order   the final norm's output bf16(x rstd g)
  size_t ssqs;         // fp32 [2L+1][d/16][Mp]   their per-16-column sums of squares
  size_t qs;           // bf16 [L][Mp][d]         queries after the rotary embedding
  size_t os;           // bf16 [L] x (Mp x d, fragment order)   attention output
  size_t hs;           // bf16 [L] x (Mp x Fp, fragment order)  SwiGLU product
  size_t attn_o;       // fp32 [H][Mp/16][KS][16][Dh]  key-split partial attention outputs
  size_t attn_ml;      // fp32 [H][Mp/16][KS][16][2]   their running max and sum
  size_t part;         // fp32 [part_slots][Mp/16][64][4]  split-K partial tiles
  size_t trace;        // int64 [G][4 + 5L][8]    phase timestamps (diagnostics)
  size_t total;
  WorkspaceLayout(const Shape& s, int max_n, int G) {
    Mp = pass_rows(max_n);
    size_t o_ = 0;
    auto take = [&](size_t bytes) {
      size_t at = o_;
      o_ = align_up(o_ + bytes, 256);
      return at;
    };
    // The regions that hold state from one pass to the next (counters, the
    // barrier, the zero line) come first, sized for the largest pass, so
    // that their offsets do not depend on the pass's node count or grid:
    // llmcad_workspace_init clears them once for every later pass.
    n_head_counters = s.H * (kMaxNodes / 16);
    n_group_counters = kPassMaxGrid;  // [O, down][up to G / 2 groups]
    counters_bytes = (size_t)(n_head_counters + 4 + n_group_counters) * 4;
    counters = take(counters_bytes);
    bar = take((size_t)kBarSlots * kBarStride * 4);
    zero = take(kZeroBytes);
    scratch_out = take((128 + 2) * 4);
    tree = take(4 * 128 * 4 + 128 * 4 * 4);
    rope = take((size_t)Mp * s.Dh * 4);
    amax = take((size_t)Mp * 4);
    lm_val = take((size_t)G * Mp * 4);
    lm_idx = take((size_t)G * Mp * 4);
    lm_sum = take((size_t)G * Mp * 4);
    xs = take((size_t)(2 * s.L + 1) * Mp * s.d * 4);
    xgs = take((size_t)(2 * s.L + 1) * Mp * s.d * 2);
    xnf = take((size_t)Mp * s.d * 2);
    ssqs = take((size_t)(2 * s.L + 1) * s.d_nb * Mp * 4);
    qs = take((size_t)s.L * Mp * s.d * 2);
    os = take((size_t)s.L * Mp * s.d * 2);
    hs = take((size_t)s.L * Mp * s.Fp * 2);
    attn_o = take((size_t)s.H * Mp * kAttnMaxSplits * s.Dh * 4);
    attn_ml = take((size_t)s.H * Mp * kAttnMaxSplits * 2 * 4);
    // split-K steps (O, down: d/16 column blocks; passes of 32 or more
    // rows) in groups of S <= kMaxSplitK workgroups: each workgroup keeps a
    // partial tile of every block of its group, G cdiv(d/16, G/S) <=
    // S d/16 + G of them
    part_slots = Mp >= 32 ? (size_t)kMaxSplitK * s.d_nb + G : 0;
    part = take(part_slots * (Mp / 16) * 1024);
    trace = take((size_t)G * pass_phases(s.L) * 8 * 8);
    total = o_;
  }
  size_t head_counters() const { return counters; }
  size_t lm_cnt() const { return head_counters() + (size_t)n_head_counters * 4; }
  size_t exit_cnt() const { return lm_cnt() + 4; }
  size_t status() const { return lm_cnt() + 8; }
  size_t group_counters() const { return lm_cnt() + 16; }
};

}  // namespace llmcad
