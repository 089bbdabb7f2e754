// Packed-weight image, GEMM work plans and workspace layout, shared by the
// host API and the kernels.  Everything here is plain integer arithmetic on
// the model shape.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "llmcad.h"

namespace llmcad {

// One packed weight block feeds one 32x32x16 MFMA: 32 output columns x 16
// inputs, bf16, 1 KiB.
constexpr int kNB = 32;                        // output columns per n-block
constexpr int kStepK = 16;                     // inputs per k-step
constexpr int kBlockBytes = kNB * kStepK * 2;  // 1 KiB
constexpr int kMaxNodes = LLMCAD_MAX_NODES;
constexpr int kAttnChunk = 128;     // key positions staged in LDS at once
constexpr int kAttnMaxSplits = 32;  // position splits per head
constexpr int kPassMaxGrid = 1024;  // workgroups of the pass
constexpr int kBarSlots = 16;       // grid-barrier counters
constexpr int kBarStride = 32;      // ints between barrier counters (128 bytes)
constexpr int kMaxCW = 16;          // n-blocks per GEMM tile at 32 rows (16 / row blocks above)
constexpr int kMaxSplits = 64;      // K splits of one GEMM
constexpr int kAStageBytes = 132 * 1024;  // LDS for one tile's activation slice
constexpr int kZeroBytes = 256 * 1024;    // zero rows the activation staging reads for padding rows

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
inline int round_up(int x, int a) { return (x + a - 1) / a * a; }
inline int cdiv(int x, int a) { return (x + a - 1) / a; }

// Rows a pass over n nodes computes: n rounded up to 32, 64 or 128 (one,
// two or four 32-row MFMA blocks).
inline int pass_rows(int n) {
  const int mb = cdiv(n, 32);
  return 32 * (mb <= 2 ? mb : 4);
}

struct Shape {
  int L, d, H, Dh, F, V;
  int Fp;      // F rounded up to 16 (SwiGLU width as stored; K of the down projection)
  int qkv_nb;  // n-blocks of the QKV projection (3d / 32)
  int d_nb;    // n-blocks of the O and down projections (d / 32)
  int gu_nb;   // n-blocks of gate/up: each holds 16 gate and the matching 16 up columns (Fp / 16)
  int v_nb;    // n-blocks of the LM head (V / 32 rounded up)
  int ks_d, ks_f;  // k-steps over d and over Fp
  explicit Shape(const llmcad_config& c)
      : L(c.n_layers), d(c.d_model), H(c.n_heads), Dh(c.head_dim), F(c.d_ffn), V(c.vocab) {
    Fp = round_up(F, 16);
    qkv_nb = 3 * d / kNB;
    d_nb = d / kNB;
    gu_nb = Fp / 16;
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

// The GEMM steps of a pass.
enum Step { STEP_QKV = 0, STEP_O = 1, STEP_GATE_UP = 2, STEP_DOWN = 3, STEP_LM = 4, kSteps = 5 };

// How one GEMM step is cut into tiles.  The n-blocks form `groups` column
// groups of cw or cw + 1 consecutive n-blocks (the first n_hi groups take
// cw + 1); each group's k-steps are cut into S slices of near-equal length.
// Tile t = (group t / S, slice t % S); workgroup g takes tiles g, g + G, ...
// A tile's activation slice sits in LDS while its weights stream through;
// the S partial results of a group are added by the workgroup that
// completes the group last.
struct GemmPlan {
  int nblocks, ksteps;
  int S, groups, cw, n_hi;
  int tiles() const { return groups * S; }
  int group_nb0(int g) const { return g * cw + (g < n_hi ? g : n_hi); }
  int group_cw(int g) const { return cw + (g < n_hi ? 1 : 0); }
  int cw_max() const { return cw + (n_hi > 0 ? 1 : 0); }
  int k0(int s) const { return (int)((long)s * ksteps / S); }
  int kt_max() const { return cdiv(ksteps, S); }
};

// Bytes of LDS a tile's bf16 activation slice takes: 1 KiB per k-step and
// 32-row block.
inline int a_stage_bytes(int kt, int mb32) { return kt * mb32 * 1024; }

// Chooses S and the column groups for G workgroups: every tile's activation
// slice must fit kAStageBytes; among those, minimise the busiest workgroup's
// weight bytes plus a share of its activation and partial-sum traffic.
inline GemmPlan plan_gemm(int nblocks, int ksteps, int mb32, int G) {
  GemmPlan best{nblocks, ksteps, 0, 0, 0, 0};
  double best_cost = 1e300;
  const int cw_cap = kMaxCW / mb32;
  for (int S = 1; S <= kMaxSplits && S <= ksteps; ++S) {
    const int kt = cdiv(ksteps, S);
    if (a_stage_bytes(kt, mb32) > kAStageBytes) continue;
    int groups = G / S;
    if (groups < 1) groups = 1;
    if (groups > nblocks) groups = nblocks;
    if (cdiv(nblocks, groups) > cw_cap) groups = cdiv(nblocks, cw_cap);
    const int cw = nblocks / groups, n_hi = nblocks % groups;
    const int cwm = cw + (n_hi > 0 ? 1 : 0);
    const int rounds = cdiv(groups * S, G);
    const double w_kb = (double)rounds * cwm * kt;
    const double a_kb = (double)rounds * a_stage_bytes(kt, mb32) / 1024.0;
    const double fix_kb = S > 1 ? (double)S * cwm * mb32 * 4.0 : 0.0;
    const double cost = w_kb + 0.5 * a_kb + 0.5 * fix_kb;
    if (cost < best_cost - 1e-9) {
      best_cost = cost;
      best = GemmPlan{nblocks, ksteps, S, groups, cw, n_hi};
    }
  }
  return best;
}

struct PassPlans {
  GemmPlan g[kSteps];
  PassPlans(const Shape& s, int mb32, int G) {
    g[STEP_QKV] = plan_gemm(s.qkv_nb, s.ks_d, mb32, G);
    g[STEP_O] = plan_gemm(s.d_nb, s.ks_d, mb32, G);
    g[STEP_GATE_UP] = plan_gemm(s.gu_nb, s.ks_d, mb32, G);
    g[STEP_DOWN] = plan_gemm(s.d_nb, s.ks_f, mb32, G);
    g[STEP_LM] = plan_gemm(s.v_nb, s.ks_d, mb32, G);
  }
  bool ok() const {
    for (int i = 0; i < kSteps; ++i)
      if (g[i].S < 1) return false;
    return true;
  }
  // fp32 words of the split-K partial buffer (shared by all steps).
  size_t part_words(int mb32) const {
    size_t m = 0;
    for (int i = 0; i < kSteps; ++i) {
      const size_t w = g[i].S > 1 ? (size_t)g[i].S * g[i].nblocks * mb32 * 1024 : 0;
      if (w > m) m = w;
    }
    return m;
  }
};

// Byte offsets inside a workspace sized for passes of up to max_n nodes on
// a device with G workgroups (row count Mp = pass_rows(max_n)).  Buffers
// handed from one phase of a pass to the next are written once per pass (one
// copy per layer), so no cache can hold a stale copy of them; buffers reused
// within a pass (partials, counters) are accessed with device-coherent
// operations only.
struct WorkspaceLayout {
  int Mp;
  int n_group_counters, n_head_counters;
  size_t counters;     // int32: groups [kSteps][max n-blocks] | heads [H] | lm | exit | status | spare
  size_t counters_bytes;
  size_t bar;          // int32 [kBarSlots][kBarStride] grid-barrier counters
  size_t scratch_out;  // int32 [128 + 2] path/len/next sink for prefill
  size_t tree;         // int32 tok[128] | parent[128] | depth[128] | pos[128] | uint32 anc[128][4]
  size_t trace;        // int64 [8][2 + 5L][8]    phase timestamps (diagnostics)
  size_t zero;         // kZeroBytes of zeros (never written by a pass)
  size_t rope;         // fp32 [Mp][Dh/2][2]      cos, sin of every node's rotary angles
  size_t amax;         // int32 [Mp]              per-node greedy token
  size_t lm_val;       // fp32 [slots][Mp]        LM-head argmax per tile (or column group)
  size_t lm_idx;       // int32 [slots][Mp]
  size_t xs;           // fp32 [2L+1][Mp][d]      residual stream versions
  size_t xgs;          // bf16 [2L+1][Mp][d]      bf16(x * g) of each version (g: its norm's gain)
  size_t ssqs;         // fp32 [2L+1][d/32][Mp]   their per-n-block sums of squares
  size_t qs;           // bf16 [L][Mp][d]         queries after the rotary embedding
  size_t os;           // bf16 [L][Mp][d]         attention output
  size_t hs;           // bf16 [L][Mp][Fp]        SwiGLU product
  size_t part;         // fp32 split-K partial tiles
  size_t attn_o;       // fp32 [H][S][Mp][Dh]     per-split unnormalised outputs
  size_t attn_ml;      // fp32 [H][S][Mp][2]      per-split running max and sum
  size_t total;
  WorkspaceLayout(const Shape& s, int max_n, int G) {
    Mp = pass_rows(max_n);
    const PassPlans plans(s, Mp / 32, G);
    size_t o_ = 0;
    auto take = [&](size_t bytes) {
      size_t at = o_;
      o_ = align_up(o_ + bytes, 256);
      return at;
    };
    int nbmax = s.v_nb;
    if (s.qkv_nb > nbmax) nbmax = s.qkv_nb;
    if (s.gu_nb > nbmax) nbmax = s.gu_nb;
    if (s.d_nb > nbmax) nbmax = s.d_nb;
    n_group_counters = kSteps * nbmax;
    n_head_counters = s.H;
    counters_bytes = (size_t)(n_group_counters + n_head_counters + 4) * 4;
    counters = take(counters_bytes);
    bar = take((size_t)kBarSlots * kBarStride * 4);
    scratch_out = take((128 + 2) * 4);
    tree = take(4 * 128 * 4 + 128 * 4 * 4);
    trace = take((size_t)8 * (2 + 5 * s.L) * 8 * 8);
    zero = take(kZeroBytes);
    rope = take((size_t)Mp * s.Dh * 4);
    amax = take((size_t)Mp * 4);
    const int lm_slots = plans.g[STEP_LM].tiles() > s.v_nb ? plans.g[STEP_LM].tiles() : s.v_nb;
    lm_val = take((size_t)lm_slots * Mp * 4);
    lm_idx = take((size_t)lm_slots * Mp * 4);
    xs = take((size_t)(2 * s.L + 1) * Mp * s.d * 4);
    xgs = take((size_t)(2 * s.L + 1) * Mp * s.d * 2);
    ssqs = take((size_t)(2 * s.L + 1) * s.d_nb * Mp * 4);
    qs = take((size_t)s.L * Mp * s.d * 2);
    os = take((size_t)s.L * Mp * s.d * 2);
    hs = take((size_t)s.L * Mp * s.Fp * 2);
    part = take(plans.part_words(Mp / 32) * 4 + 256);
    attn_o = take((size_t)s.H * kAttnMaxSplits * Mp * s.Dh * 4);
    attn_ml = take((size_t)s.H * kAttnMaxSplits * Mp * 2 * 4);
    total = o_;
  }
  size_t group_counters(int step) const { return counters + (size_t)step * (n_group_counters / kSteps) * 4; }
  size_t head_counters() const { return counters + (size_t)n_group_counters * 4; }
  size_t lm_cnt() const { return head_counters() + (size_t)n_head_counters * 4; }
  size_t exit_cnt() const { return lm_cnt() + 4; }
  size_t status() const { return lm_cnt() + 8; }
};

}  // namespace llmcad
