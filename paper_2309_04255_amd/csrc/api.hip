// Host side of the C ABI: argument checks, packing, launch sequencing.
//
// A verification pass (§3.2, "Batched non-autoregressive verification" and
// "Depth-first verified sequence searching") is enqueued as
//   embed+tree prep, then per layer: QKV GEMM (RMSNorm prologue, rotary +
//   KV-write epilogue) -> tree attention -> O GEMM (+residual) -> gate/up GEMM
//   (RMSNorm prologue, SwiGLU epilogue) -> down GEMM (+residual),
//   then the LM-head GEMM (final RMSNorm prologue, argmax epilogue) whose last
//   workgroup performs the accept walk.
// Prefill runs the same sequence on chains of tokens (a chain's ancestor mask
// is the causal mask and its depth is its offset).
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>

#include "kernels.h"
#include "layout.h"
#include "llmcad.h"

using namespace llmcad;

namespace {

int env_int(const char* name, int dflt) {
  const char* v = getenv(name);
  if (v == nullptr || *v == 0) return dflt;
  int x = atoi(v);
  return x > 0 ? x : dflt;
}

int check_cfg(const llmcad_config* c) {
  if (c == nullptr) return LLMCAD_EARG;
  if (c->n_layers < 1 || c->d_model < 1 || c->n_heads < 1 || c->head_dim < 1 || c->d_ffn < 1 ||
      c->vocab < 1)
    return LLMCAD_EARG;
  if (!(c->rms_eps > 0.0f) || !(c->rope_theta > 1.0f)) return LLMCAD_EARG;
  if (c->head_dim != 64 && c->head_dim != 128) return LLMCAD_ESHAPE;
  if ((long)c->n_heads * c->head_dim != c->d_model) return LLMCAD_ESHAPE;
  if (c->d_model % 64 != 0) return LLMCAD_ESHAPE;
  if (c->n_layers > 4096 || c->d_model > 65536 || c->d_ffn > (1 << 20) || c->vocab > (1 << 24))
    return LLMCAD_ESHAPE;
  if (c->weight_bits != 0 && c->weight_bits != 16 && c->weight_bits != 4) return LLMCAD_EARG;
  if (c->weight_bits == 4 && (c->d_model % kQ4Group != 0 || c->d_ffn % kQ4Group != 0)) return LLMCAD_ESHAPE;
  return LLMCAD_OK;
}

hipError_t g_last_error = hipSuccess;

// Diagnostics: optional HIP event pairs around every launch of one kernel
// class (see llmcad_timing_enable).  Not used unless enabled.
struct Timing {
  int kclass = -1;
  int capacity = 0;
  int used = 0;
  hipEvent_t* ev = nullptr;  // [capacity][2]
} g_timing;

struct TimedLaunch {
  bool on;
  hipStream_t st;
  int slot;
  TimedLaunch(int kclass, hipStream_t s) : on(false), st(s), slot(-1) {
    if (g_timing.kclass == kclass && g_timing.used < g_timing.capacity) {
      on = true;
      slot = g_timing.used++;
      (void)hipEventRecord(g_timing.ev[2 * slot], st);
    }
  }
  ~TimedLaunch() {
    if (on) (void)hipEventRecord(g_timing.ev[2 * slot + 1], st);
  }
};

#define HIP_TRY(expr)                 \
  do {                                \
    hipError_t e_ = (expr);           \
    if (e_ != hipSuccess) {           \
      g_last_error = e_;              \
      return LLMCAD_EHIP;             \
    }                                 \
  } while (0)

struct Pass {
  const llmcad_config* cfg;
  const char* packed;
  char* k_cache;
  char* v_cache;
  int cap;
  int prefix_len;
  int n;       // rows: nodes [m0, m0 + n) of a tree of nt nodes
  int m0 = 0;
  int nt = 0;  // (0: n)
  float* logits;
  int row_lo;
  int* path;
  int* accept_len;
  int* next_token;
  char* ws;
  hipStream_t st;
  llmcad_candidates* cand = nullptr;  // candidate summaries of the computed rows, or null
  float cand_thr = 0.0f;
};

// Device facts for the pass, looked up once per device.
struct DeviceInfo {
  int cus = 0;
};
DeviceInfo device_info() {
  static DeviceInfo cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return DeviceInfo();
  if (cache[dev].cus == 0) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess)
      cache[dev].cus = cus;
  }
  return cache[dev];
}

// Workgroups of a pass on the current device: one per CU, at most
// kPassMaxGrid; LLMCAD_PASS_GRID (diagnostics) asks for fewer.  Without a
// device (sizing on a host with no GPU) the MI355X count, 256, stands in.
int pass_grid() {
  const DeviceInfo dev = device_info();
  int G = dev.cus > 0 ? dev.cus : 256;
  const int want = env_int("LLMCAD_PASS_GRID", 0);
  if (want > 0 && want < G) G = want;
  return G > kPassMaxGrid ? kPassMaxGrid : G;
}

// Runs of more than 8 gate/up blocks per workgroup at 16 or 32 rows (the
// 30B shape: 8.75) take one tile of 9 instead of 8 + 1, whose lone block
// re-reads the whole activation matrix (-2.5% per 30B pass): the pass then
// runs the kernel instance with wide gate/up tiles.
bool gate_up_wide(const Shape& s, int Mp, int G) {
  return Mp <= 32 && !s.q4 && cdiv(step_blocks(s, STEP_GATE_UP), G) > 8;
}

int run_pass(const Pass& a, const TreeArgs& tree) {
  const Shape s(*a.cfg);
  const PackedLayout P(s);
  const int G = pass_grid();
  const WorkspaceLayout W(s, a.n, G);
  const int MB = W.Mp / 16;
  const bool wide = gate_up_wide(s, W.Mp, G);
  const int occ = pass_occupancy(MB, s.Dh, wide);
  if (device_info().cus <= 0 || occ * device_info().cus < G) {
    g_last_error = hipErrorInvalidConfiguration;
    return LLMCAD_EHIP;
  }
  char* ws = a.ws;

  PassParams p;
  memset(&p, 0, sizeof(p));
  p.magic = kPassMagic;
  p.L = s.L;
  p.d = s.d;
  p.H = s.H;
  p.Dh = s.Dh;
  p.F = s.F;
  p.Fp = s.Fp;
  p.V = s.V;
  p.eps = a.cfg->rms_eps;
  p.inv_d = 1.0f / (float)s.d;
  p.log2_theta = (float)log2((double)a.cfg->rope_theta);
  p.scale_log2 = (float)(1.4426950408889634 / sqrt((double)s.Dh));
  p.n = a.n;
  p.m0 = a.m0;
  p.nt = a.nt > 0 ? a.nt : a.n;
  p.Mp = W.Mp;
  p.prefix_len = a.prefix_len;
  p.cap = a.cap;
  p.G = G;
  p.packed = a.packed;
  p.o_embed = (long long)P.embed;
  p.o_final_norm = (long long)P.final_norm;
  p.layer0 = (long long)P.globals_end;
  p.layer_bytes = (long long)P.layer_bytes;
  p.o_attn_norm = (long long)P.attn_norm;
  p.o_ffn_norm = (long long)P.ffn_norm;
  p.d_nb = s.d_nb;
  const long long w_off[kSteps] = {(long long)P.w_qkv, (long long)P.w_o, (long long)P.w_gate_up,
                                   (long long)P.w_down, (long long)P.lm_head};
  for (int i = 0; i < kSteps; ++i) {
    StepPlan& sp = p.step[i];
    sp.nblocks = step_blocks(s, i);
    sp.layer_rel = i == STEP_LM ? 0 : 1;
    sp.q4 = s.q4 && i != STEP_LM ? 1 : 0;
    // bf16: k-steps of 32 inputs; 4-bit: scale groups of 128 inputs
    sp.ksteps = sp.q4 ? step_groups(s, i) : step_ksteps(s, i);
    sp.w_off = w_off[i];
    sp.s_off = sp.q4 ? w_off[i] + (long long)q4_codes_bytes(sp.nblocks, sp.ksteps) : 0;
    sp.split = 1;
    sp.wide = i == STEP_GATE_UP && wide ? 1 : 0;
  }
  // Split-K for the projections with one column block per workgroup (O and
  // down: d/16 blocks): groups of S workgroups share a group's blocks, each
  // over 1/S of the k-steps, so each reads 1/S of the activations per block
  // of weights; the partial tiles meet in memory and each workgroup finishes
  // 1/S of the group's blocks.  It pays where the activations outweigh the
  // weights by far: the down projection (K = F) of passes of 64 or more rows,
  // in pairs (measured at the LLaMA-7B shape: -3.5% per pass at 41 and 128
  // rows; at 32 rows, and for O, the hand-off costs more than it saves).
  // (LLMCAD_SPLIT_O / LLMCAD_SPLIT_DOWN, diagnostics, ask for 1, 2 or 4.)
  {
    const int want[2] = {env_int("LLMCAD_SPLIT_O", 1), env_int("LLMCAD_SPLIT_DOWN", W.Mp >= 64 ? 2 : 1)};
    const int steps[2] = {STEP_O, STEP_DOWN};
    for (int j = 0; j < 2; ++j) {
      StepPlan& sp = p.step[steps[j]];
      const int S = want[j];
      if ((S == 2 || S == 4) && !sp.q4 && G % S == 0 && sp.nblocks >= G / S &&
          (size_t)G * cdiv(sp.nblocks, G / S) <= W.part_slots)
        sp.split = S;
    }
  }
  p.k_cache = (bf16*)a.k_cache;
  p.v_cache = (bf16*)a.v_cache;
  p.tree = (int*)(ws + W.tree);
  p.zero = ws + W.zero;
  p.rope = (float*)(ws + W.rope);
  p.x = (float*)(ws + W.xs);
  p.xg = (bf16*)(ws + W.xgs);
  p.xnf = (bf16*)(ws + W.xnf);
  p.ssq = (float*)(ws + W.ssqs);
  p.ssq_regs = W.Mp <= 32 && cdiv(s.d_nb, 1024 / W.Mp) <= 8 ? 1 : 0;
  p.q = (bf16*)(ws + W.qs);
  p.o = (bf16*)(ws + W.os);
  p.h = (bf16*)(ws + W.hs);
  // Key splits per (head, row block) of the attention: about four 32-key
  // steps of the prefix per split (one per wave), at most four splits
  // (LLMCAD_ATTN_SPLITS, diagnostics, asks for 1 to 4).  A workgroup pulls its
  // keys and values at the rate one CU's memory path gives, so a head's keys
  // are spread over several; the splits' merge costs a hand-off through memory.
  // Fewer splits when the (head, row block) pairs alone fill the grid: each
  // split of a pair re-reads the keys and values the pair's other row blocks
  // read too, and another round of units costs more than a longer unit.
  const int prefix_steps = cdiv(a.prefix_len, 32);
  const int pairs = s.H * cdiv(a.n, 16);
  int KS = cdiv(prefix_steps, 4);
  if (KS > G / pairs) KS = G / pairs;
  KS = env_int("LLMCAD_ATTN_SPLITS", KS);
  if (KS > kAttnMaxSplits) KS = kAttnMaxSplits;
  if (KS > prefix_steps) KS = prefix_steps;
  if (KS < 1) KS = 1;
  p.attn_splits = KS;
  p.attn_o = (float*)(ws + W.attn_o);
  p.attn_ml = (float*)(ws + W.attn_ml);
  p.head_cnt = (int*)(ws + W.head_counters());
  p.part = (float*)(ws + W.part);
  p.grp_cnt = (int*)(ws + W.group_counters());
  p.lm_cnt = (int*)(ws + W.lm_cnt());
  p.exit_cnt = (int*)(ws + W.exit_cnt());
  p.status = (int*)(ws + W.status());
  p.bar = (int*)(ws + W.bar);
  p.lm_val = (float*)(ws + W.lm_val);
  p.lm_idx = (int*)(ws + W.lm_idx);
  p.lm_sum = (float*)(ws + W.lm_sum);
  p.cand = a.cand;
  p.cand_thr = a.cand_thr;
  p.amax = (int*)(ws + W.amax);
  p.logits = a.logits;
  p.row_lo = a.row_lo;
  p.path = a.path;
  p.accept_len = a.accept_len;
  p.next_token = a.next_token;
  p.spin_limit = env_int("LLMCAD_SPIN_LIMIT", 4000000);
  // (diagnostics, for tests of the failure path: every grid wait gives up at
  // once, so the pass ends with status 1 and every workgroup exits normally)
  if (env_int("LLMCAD_FAIL_WAITS", 0) == 1) p.spin_limit = -1;
  // (diagnostics: a smaller pre-barrier copy, for every step or for one:
  // LLMCAD_WL_STAGES_QKV / _O / _GU / _DOWN / _LM)
  {
    const int all = env_int("LLMCAD_WL_STAGES", 1 << 20);
    const char* names[kSteps] = {"LLMCAD_WL_STAGES_QKV", "LLMCAD_WL_STAGES_O", "LLMCAD_WL_STAGES_GU",
                                 "LLMCAD_WL_STAGES_DOWN", "LLMCAD_WL_STAGES_LM"};
    for (int i = 0; i < kSteps; ++i) p.step[i].wl_cap = env_int(names[i], all);
  }
  // (diagnostics: LLMCAD_ATTN_PREFETCH=2 fetches every attention step after the barrier)
  p.attn_prefetch = env_int("LLMCAD_ATTN_PREFETCH", 1) == 2 ? 0 : 1;
  // (diagnostics: LLMCAD_ROW_TILES=2 turns the row-split tiles off)
  p.row_tiles = env_int("LLMCAD_ROW_TILES", 1) == 2 ? 0 : 1;
  p.trace = env_int("LLMCAD_TRACE", 0) ? (long long*)(ws + W.trace) : nullptr;
  TimedLaunch tl(LLMCAD_KERNEL_PASS, a.st);
  HIP_TRY(launch_pass(MB, p, tree, a.st));
  return LLMCAD_OK;
}

// The workspace of llmcad_verify_tree_noalloc: device memory the library
// holds itself, one copy per device (each device that runs the entry point
// holds it until the process ends).  In host code `scratch` names a host-side
// stand-in, not the device array: its device address is looked up once per
// device (scratch_base) and only that address is handed to the kernels.
static __device__ __align__(256) char scratch[LLMCAD_SCRATCH_BYTES];

// Device address of this device's `scratch` (null if the lookup failed; the
// HIP status is kept for llmcad_status_string).
char* scratch_base() {
  static std::mutex mu;
  static char* base[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0 || dev >= 64) {
    g_last_error = e != hipSuccess ? e : hipErrorInvalidDevice;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (base[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr) {
      g_last_error = e != hipSuccess ? e : hipErrorInvalidSymbol;
      return nullptr;
    }
    base[dev] = (char*)p;
  }
  return base[dev];
}

// Host-side checks of a verification pass's arguments (llmcad_verify_tree's
// contract), then the tree copied into the launch arguments.
int check_verify_args(const llmcad_config* cfg, const void* packed, const void* k_cache, const void* v_cache,
                      int32_t capacity, int32_t prefix_len, const int32_t* tree_tokens, const int32_t* parent,
                      int32_t n, const int32_t* path, const int32_t* accept_len, const int32_t* next_token,
                      TreeArgs* tree) {
  int rc = check_cfg(cfg);
  if (rc != LLMCAD_OK) return rc;
  if (!packed || !k_cache || !v_cache || !tree_tokens || !parent || !path || !accept_len || !next_token)
    return LLMCAD_EARG;
  if (n < 1 || n > kMaxNodes) return LLMCAD_ETREE;
  if (parent[0] != -1) return LLMCAD_ETREE;
  for (int i = 0; i < n; ++i) {
    if (tree_tokens[i] < 0 || tree_tokens[i] >= cfg->vocab) return LLMCAD_ETREE;
    if (i > 0 && (parent[i] < 0 || parent[i] >= i)) return LLMCAD_ETREE;
  }
  if (capacity < 64 || capacity % 64 != 0 || prefix_len < 0 || (long)prefix_len + n > capacity)
    return LLMCAD_ECAPACITY;
  memset(tree, 0, sizeof(*tree));
  for (int i = 0; i < n; ++i) {
    tree->tok[i] = tree_tokens[i];
    tree->parent[i] = parent[i];
  }
  return LLMCAD_OK;
}

}  // namespace

extern "C" {

int llmcad_check_config(const llmcad_config* cfg) { return check_cfg(cfg); }

size_t llmcad_packed_bytes(const llmcad_config* cfg) {
  if (check_cfg(cfg) != LLMCAD_OK) return 0;
  return PackedLayout(Shape(*cfg)).total;
}

int llmcad_pack_globals(const llmcad_config* cfg, const void* tok_embed, const void* final_norm,
                        const void* lm_head, void* packed, size_t packed_bytes, void* stream) {
  int rc = check_cfg(cfg);
  if (rc != LLMCAD_OK) return rc;
  if (!tok_embed || !final_norm || !lm_head || !packed) return LLMCAD_EARG;
  const Shape s(*cfg);
  const PackedLayout P(s);
  if (packed_bytes < P.total) return LLMCAD_EWORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  char* out = (char*)packed;
  HIP_TRY(hipMemcpyAsync(out + P.embed, tok_embed, (size_t)s.V * s.d * 2, hipMemcpyDeviceToDevice, st));
  HIP_TRY(hipMemcpyAsync(out + P.final_norm, final_norm, (size_t)s.d * 2, hipMemcpyDeviceToDevice, st));
  HIP_TRY(launch_pack(lm_head, s.V, s.d, out + P.lm_head, s.v_nb, s.ks_d, PACK_PLAIN, s.F, st));
  return LLMCAD_OK;
}

int llmcad_pack_layer(const llmcad_config* cfg, int32_t layer, const llmcad_layer_weights* src,
                      void* packed, size_t packed_bytes, void* stream) {
  int rc = check_cfg(cfg);
  if (rc != LLMCAD_OK) return rc;
  if (!src || !packed || layer < 0 || layer >= cfg->n_layers || cfg->weight_bits == 4) return LLMCAD_EARG;
  if (!src->attn_norm || !src->w_qkv || !src->w_o || !src->ffn_norm || !src->w_gate_up ||
      !src->w_down)
    return LLMCAD_EARG;
  const Shape s(*cfg);
  const PackedLayout P(s);
  if (packed_bytes < P.total) return LLMCAD_EWORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  char* out = (char*)packed + P.layer(layer);
  HIP_TRY(hipMemcpyAsync(out + P.attn_norm, src->attn_norm, (size_t)s.d * 2, hipMemcpyDeviceToDevice, st));
  HIP_TRY(hipMemcpyAsync(out + P.ffn_norm, src->ffn_norm, (size_t)s.d * 2, hipMemcpyDeviceToDevice, st));
  HIP_TRY(launch_pack(src->w_qkv, 3 * s.d, s.d, out + P.w_qkv, s.qkv_nb, s.ks_d, PACK_QKV_ROPE, s.Dh,
                      st));
  HIP_TRY(launch_pack(src->w_o, s.d, s.d, out + P.w_o, s.d_nb, s.ks_d, PACK_PLAIN, s.F, st));
  HIP_TRY(launch_pack(src->w_gate_up, 2 * s.F, s.d, out + P.w_gate_up, s.gu_nb, s.ks_d, PACK_GATE_UP,
                      s.F, st));
  HIP_TRY(launch_pack(src->w_down, s.d, s.F, out + P.w_down, s.d_nb, s.ks_f, PACK_PLAIN, s.F, st));
  return LLMCAD_OK;
}

int llmcad_pack_layer_q4(const llmcad_config* cfg, int32_t layer, const llmcad_q4_layer_weights* src,
                         void* packed, size_t packed_bytes, void* stream) {
  int rc = check_cfg(cfg);
  if (rc != LLMCAD_OK) return rc;
  if (!src || !packed || layer < 0 || layer >= cfg->n_layers || cfg->weight_bits != 4) return LLMCAD_EARG;
  const llmcad_q4_matrix* m[4] = {&src->w_qkv, &src->w_o, &src->w_gate_up, &src->w_down};
  if (!src->attn_norm || !src->ffn_norm) return LLMCAD_EARG;
  for (int i = 0; i < 4; ++i)
    if (!m[i]->codes || !m[i]->scales) return LLMCAD_EARG;
  const Shape s(*cfg);
  const PackedLayout P(s);
  if (packed_bytes < P.total) return LLMCAD_EWORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  char* out = (char*)packed + P.layer(layer);
  HIP_TRY(hipMemcpyAsync(out + P.attn_norm, src->attn_norm, (size_t)s.d * 2, hipMemcpyDeviceToDevice, st));
  HIP_TRY(hipMemcpyAsync(out + P.ffn_norm, src->ffn_norm, (size_t)s.d * 2, hipMemcpyDeviceToDevice, st));
  // (N rows, K inputs, blocks, groups, column order, its parameter, offset)
  struct Mat {
    int N, K, nb, gs, kind, aux;
    size_t off;
  } mats[4] = {
      {3 * s.d, s.d, s.qkv_nb, s.gs_d, PACK_QKV_ROPE, s.Dh, P.w_qkv},
      {s.d, s.d, s.d_nb, s.gs_d, PACK_PLAIN, s.F, P.w_o},
      {2 * s.F, s.d, s.gu_nb, s.gs_d, PACK_GATE_UP, s.F, P.w_gate_up},
      {s.d, s.F, s.d_nb, s.gs_f, PACK_PLAIN, s.F, P.w_down},
  };
  for (int i = 0; i < 4; ++i) {
    const Mat& q = mats[i];
    HIP_TRY(launch_pack_q4(m[i]->codes, m[i]->scales, q.N, q.K, out + q.off, out + q.off + q4_codes_bytes(q.nb, q.gs),
                           q.nb, q.gs, q.kind, q.aux, st));
  }
  return LLMCAD_OK;
}

size_t llmcad_workspace_bytes(const llmcad_config* cfg, int32_t max_n) {
  if (check_cfg(cfg) != LLMCAD_OK || max_n < 1 || max_n > kMaxNodes) return 0;
  return WorkspaceLayout(Shape(*cfg), max_n, pass_grid()).total;
}

int llmcad_workspace_init(const llmcad_config* cfg, int32_t max_n, void* workspace,
                          size_t workspace_bytes, void* stream) {
  int rc = check_cfg(cfg);
  if (rc != LLMCAD_OK) return rc;
  if (!workspace || max_n < 1 || max_n > kMaxNodes) return LLMCAD_EARG;
  const WorkspaceLayout W(Shape(*cfg), max_n, pass_grid());
  if (workspace_bytes < W.total) return LLMCAD_EWORKSPACE;
  HIP_TRY(hipMemsetAsync((char*)workspace + W.counters, 0, W.counters_bytes, (hipStream_t)stream));
  HIP_TRY(hipMemsetAsync((char*)workspace + W.zero, 0, kZeroBytes, (hipStream_t)stream));
  HIP_TRY(hipMemsetAsync((char*)workspace + W.bar, 0, (size_t)kBarSlots * kBarStride * 4,
                          (hipStream_t)stream));
  return LLMCAD_OK;
}

int llmcad_verify_tree(const llmcad_config* cfg, const void* packed, void* k_cache, void* v_cache,
                       int32_t capacity, int32_t prefix_len, const int32_t* tree_tokens,
                       const int32_t* parent, int32_t n, float* logits, int32_t* path,
                       int32_t* accept_len, int32_t* next_token, void* workspace,
                       size_t workspace_bytes, void* stream) {
  TreeArgs tree;
  int rc = check_verify_args(cfg, packed, k_cache, v_cache, capacity, prefix_len, tree_tokens, parent, n, path,
                             accept_len, next_token, &tree);
  if (rc != LLMCAD_OK) return rc;
  if (!workspace) return LLMCAD_EARG;
  const Shape s(*cfg);
  if (workspace_bytes < WorkspaceLayout(s, n, pass_grid()).total) return LLMCAD_EWORKSPACE;
  Pass a;
  a.cfg = cfg;
  a.packed = (const char*)packed;
  a.k_cache = (char*)k_cache;
  a.v_cache = (char*)v_cache;
  a.cap = capacity;
  a.prefix_len = prefix_len;
  a.n = n;
  a.logits = logits;
  a.row_lo = 0;
  a.path = path;
  a.accept_len = accept_len;
  a.next_token = next_token;
  a.ws = (char*)workspace;
  a.st = (hipStream_t)stream;
  return run_pass(a, tree);
}

int llmcad_verify_tree_noalloc(const llmcad_config* cfg, const void* packed, void* k_cache, void* v_cache,
                               int32_t capacity, int32_t prefix_len, const int32_t* tree_tokens,
                               const int32_t* parent, int32_t n, float* logits, int32_t* path,
                               int32_t* accept_len, int32_t* next_token, int32_t* status, void* stream) {
  TreeArgs tree;
  int rc = check_verify_args(cfg, packed, k_cache, v_cache, capacity, prefix_len, tree_tokens, parent, n, path,
                             accept_len, next_token, &tree);
  if (rc != LLMCAD_OK) return rc;
  const Shape s(*cfg);
  const WorkspaceLayout W(s, n, pass_grid());
  if (W.total > (size_t)LLMCAD_SCRATCH_BYTES) return LLMCAD_EWORKSPACE;
  char* ws = scratch_base();
  if (ws == nullptr) return LLMCAD_EHIP;
  hipStream_t st = (hipStream_t)stream;
  // The scratch keeps the previous call's contents: its synchronisation
  // state (counters with the pass status, barrier counters, the zero line,
  // which lie first and together) starts every call cleared.
  HIP_TRY(hipMemsetAsync(ws, 0, W.zero + kZeroBytes, st));
  Pass a;
  a.cfg = cfg;
  a.packed = (const char*)packed;
  a.k_cache = (char*)k_cache;
  a.v_cache = (char*)v_cache;
  a.cap = capacity;
  a.prefix_len = prefix_len;
  a.n = n;
  a.logits = logits;
  a.row_lo = 0;
  a.path = path;
  a.accept_len = accept_len;
  a.next_token = next_token;
  a.ws = ws;
  a.st = st;
  rc = run_pass(a, tree);
  if (rc != LLMCAD_OK) return rc;
  if (status != nullptr) HIP_TRY(hipMemcpyAsync(status, ws + W.status(), 4, hipMemcpyDeviceToDevice, st));
  return LLMCAD_OK;
}

}  // extern "C"

namespace {

static_assert(sizeof(llmcad_candidates) == (4 + 2 * LLMCAD_CAND_MAX) * 4, "candidate record layout");

// llmcad_extend_tree, and with `cand` its candidate-summary variant.
int extend_tree(const llmcad_config* cfg, const void* packed, void* k_cache, void* v_cache, int32_t capacity,
                int32_t prefix_len, const int32_t* tree_tokens, const int32_t* parent, int32_t n, int32_t first,
                float* logits, llmcad_candidates* cand, float threshold, void* workspace, size_t workspace_bytes,
                void* stream) {
  int rc = check_cfg(cfg);
  if (rc != LLMCAD_OK) return rc;
  if (!packed || !k_cache || !v_cache || !tree_tokens || !parent || !workspace) return LLMCAD_EARG;
  if (n < 1 || n > kMaxNodes || first < 0 || first >= n) return LLMCAD_ETREE;
  if (parent[0] != -1) return LLMCAD_ETREE;
  for (int i = 0; i < n; ++i) {
    if (tree_tokens[i] < 0 || tree_tokens[i] >= cfg->vocab) return LLMCAD_ETREE;
    if (i > 0 && (parent[i] < 0 || parent[i] >= i)) return LLMCAD_ETREE;
  }
  if (capacity < 64 || capacity % 64 != 0 || prefix_len < 0 || (long)prefix_len + n > capacity)
    return LLMCAD_ECAPACITY;
  const Shape s(*cfg);
  const int G = pass_grid();
  if (workspace_bytes < WorkspaceLayout(s, n - first, G).total) return LLMCAD_EWORKSPACE;
  TreeArgs tree;
  memset(&tree, 0, sizeof(tree));
  for (int i = 0; i < n; ++i) {
    tree.tok[i] = tree_tokens[i];
    tree.parent[i] = parent[i];
  }
  int* sink = (int*)((char*)workspace + WorkspaceLayout(s, 1, G).scratch_out);  // (no walk is run)
  Pass a;
  a.cfg = cfg;
  a.packed = (const char*)packed;
  a.k_cache = (char*)k_cache;
  a.v_cache = (char*)v_cache;
  a.cap = capacity;
  a.prefix_len = prefix_len;
  a.n = n - first;
  a.m0 = first;
  a.nt = n;
  a.logits = logits;
  a.row_lo = 0;
  a.path = sink;
  a.accept_len = sink + 128;
  a.next_token = sink + 129;
  a.ws = (char*)workspace;
  a.st = (hipStream_t)stream;
  a.cand = cand;
  a.cand_thr = threshold;
  return run_pass(a, tree);
}

}  // namespace

extern "C" {

int llmcad_extend_tree(const llmcad_config* cfg, const void* packed, void* k_cache, void* v_cache,
                       int32_t capacity, int32_t prefix_len, const int32_t* tree_tokens, const int32_t* parent,
                       int32_t n, int32_t first, float* logits, void* workspace, size_t workspace_bytes,
                       void* stream) {
  return extend_tree(cfg, packed, k_cache, v_cache, capacity, prefix_len, tree_tokens, parent, n, first, logits,
                     nullptr, 0.0f, workspace, workspace_bytes, stream);
}

int llmcad_extend_tree_candidates(const llmcad_config* cfg, const void* packed, void* k_cache, void* v_cache,
                                  int32_t capacity, int32_t prefix_len, const int32_t* tree_tokens,
                                  const int32_t* parent, int32_t n, int32_t first, float threshold, float* logits,
                                  llmcad_candidates* cand, void* workspace, size_t workspace_bytes, void* stream) {
  const int rc = check_cfg(cfg);
  if (rc != LLMCAD_OK) return rc;
  if (!logits || !cand || !(threshold > 0.0f && threshold < 1.0f)) return LLMCAD_EARG;
  return extend_tree(cfg, packed, k_cache, v_cache, capacity, prefix_len, tree_tokens, parent, n, first, logits,
                     cand, threshold, workspace, workspace_bytes, stream);
}

int llmcad_commit_path(const llmcad_config* cfg, void* k_cache, void* v_cache, int32_t capacity,
                       int32_t prefix_len, const int32_t* path, const int32_t* accept_len, int32_t n,
                       void* stream) {
  int rc = check_cfg(cfg);
  if (rc != LLMCAD_OK) return rc;
  if (!k_cache || !v_cache || !path || !accept_len) return LLMCAD_EARG;
  if (n < 1 || n > kMaxNodes) return LLMCAD_ETREE;
  if (capacity < 64 || capacity % 64 != 0 || prefix_len < 0 || (long)prefix_len + n > capacity)
    return LLMCAD_ECAPACITY;
  if (n == 1) return LLMCAD_OK;  // only the root, already in place
  HIP_TRY(launch_commit(k_cache, v_cache, cfg->n_layers * cfg->n_heads, capacity, prefix_len, path, accept_len, n,
                        cfg->head_dim, (hipStream_t)stream));
  return LLMCAD_OK;
}

int llmcad_prefill(const llmcad_config* cfg, const void* packed, void* k_cache, void* v_cache,
                   int32_t capacity, const int32_t* tokens, int32_t n_tokens, int32_t start_pos,
                   float* last_logits, void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_cfg(cfg);
  if (rc != LLMCAD_OK) return rc;
  if (!packed || !k_cache || !v_cache || !tokens || !workspace) return LLMCAD_EARG;
  if (n_tokens < 1) return LLMCAD_ETREE;
  for (int i = 0; i < n_tokens; ++i)
    if (tokens[i] < 0 || tokens[i] >= cfg->vocab) return LLMCAD_ETREE;
  if (capacity < 64 || capacity % 64 != 0 || start_pos < 0 || (long)start_pos + n_tokens > capacity)
    return LLMCAD_ECAPACITY;
  const Shape s(*cfg);
  // Largest chain the workspace holds.
  int chunk = 0;
  const int G = pass_grid();
  for (int m = kMaxNodes; m >= 1; --m)
    if (WorkspaceLayout(s, m, G).total <= workspace_bytes) {
      chunk = m;
      break;
    }
  if (chunk == 0) return LLMCAD_EWORKSPACE;
  const WorkspaceLayout W(s, 1, G);
  int* sink = (int*)((char*)workspace + W.scratch_out);  // path/len/next are not needed
  for (int off = 0; off < n_tokens; off += chunk) {
    const int len = (n_tokens - off) < chunk ? (n_tokens - off) : chunk;
    TreeArgs tree;
    memset(&tree, 0, sizeof(tree));
    for (int i = 0; i < len; ++i) {
      tree.tok[i] = tokens[off + i];
      tree.parent[i] = i - 1;
    }
    const bool last = off + len == n_tokens;
    Pass a;
    a.cfg = cfg;
    a.packed = (const char*)packed;
    a.k_cache = (char*)k_cache;
    a.v_cache = (char*)v_cache;
    a.cap = capacity;
    a.prefix_len = start_pos + off;
    a.n = len;
    a.logits = last ? last_logits : nullptr;
    a.row_lo = len - 1;
    a.path = sink;
    a.accept_len = sink + 128;
    a.next_token = sink + 129;
    a.ws = (char*)workspace;
    a.st = (hipStream_t)stream;
    rc = run_pass(a, tree);
    if (rc != LLMCAD_OK) return rc;
  }
  return LLMCAD_OK;
}

int llmcad_timing_enable(int32_t kernel_class, int32_t max_launches) {
  if (g_timing.ev != nullptr) {
    for (int i = 0; i < 2 * g_timing.capacity; ++i) (void)hipEventDestroy(g_timing.ev[i]);
    free(g_timing.ev);
    g_timing = Timing();
  }
  if (kernel_class < 0) return LLMCAD_OK;
  if (kernel_class > LLMCAD_KERNEL_PASS || max_launches < 1) return LLMCAD_EARG;
  g_timing.ev = (hipEvent_t*)calloc((size_t)2 * max_launches, sizeof(hipEvent_t));
  if (g_timing.ev == nullptr) return LLMCAD_EARG;
  for (int i = 0; i < 2 * max_launches; ++i) {
    hipError_t e = hipEventCreate(&g_timing.ev[i]);
    if (e != hipSuccess) {
      g_last_error = e;
      g_timing.capacity = i / 2;
      return LLMCAD_EHIP;
    }
  }
  g_timing.capacity = max_launches;
  g_timing.kclass = kernel_class;
  return LLMCAD_OK;
}

int llmcad_timing_read(int32_t kernel_class, double* total_ms, int32_t* launches) {
  if (!total_ms || !launches) return LLMCAD_EARG;
  *total_ms = 0.0;
  *launches = 0;
  if (kernel_class != g_timing.kclass) return LLMCAD_OK;
  double sum = 0.0;
  for (int i = 0; i < g_timing.used; ++i) {
    HIP_TRY(hipEventSynchronize(g_timing.ev[2 * i + 1]));
    float ms = 0.0f;
    HIP_TRY(hipEventElapsedTime(&ms, g_timing.ev[2 * i], g_timing.ev[2 * i + 1]));
    sum += ms;
  }
  *total_ms = sum;
  *launches = g_timing.used;
  g_timing.used = 0;
  return LLMCAD_OK;
}

const char* llmcad_status_string(int status) {
  switch (status) {
    case LLMCAD_OK: return "ok";
    case LLMCAD_EARG: return "invalid argument";
    case LLMCAD_ETREE: return "invalid token tree";
    case LLMCAD_ECAPACITY: return "KV cache capacity exceeded";
    case LLMCAD_ESHAPE: return "unsupported model shape";
    case LLMCAD_EHIP: return hipGetErrorString(g_last_error);
    case LLMCAD_EWORKSPACE: return "workspace or packed image too small";
    default: return "unknown status";
  }
}

int llmcad_workspace_region(const llmcad_config* cfg, int32_t max_n, int32_t which, size_t* offset,
                            size_t* bytes) {
  int rc = check_cfg(cfg);
  if (rc != LLMCAD_OK) return rc;
  if (!offset || !bytes || max_n < 1 || max_n > kMaxNodes) return LLMCAD_EARG;
  const Shape s(*cfg);
  const WorkspaceLayout W(s, max_n, pass_grid());
  switch (which) {
    case 0: *offset = W.xs + (size_t)2 * s.L * W.Mp * s.d * 4; *bytes = (size_t)W.Mp * s.d * 4; break;
    case 1: *offset = W.qs; *bytes = (size_t)W.Mp * s.d * 2; break;
    case 2: *offset = W.os; *bytes = (size_t)W.Mp * s.d * 2; break;
    case 3: *offset = W.hs; *bytes = (size_t)W.Mp * s.Fp * 2; break;
    case 4: *offset = W.amax; *bytes = (size_t)W.Mp * 4; break;
    case 5: *offset = W.status(); *bytes = 4; break;
    case 6: *offset = W.trace; *bytes = (size_t)pass_grid() * pass_phases(s.L) * 8 * 8; break;
    case 7: *offset = W.xs; *bytes = (size_t)(2 * s.L + 1) * W.Mp * s.d * 4; break;
    case 8: *offset = W.ssqs; *bytes = (size_t)(2 * s.L + 1) * s.d_nb * W.Mp * 4; break;
    case 9: *offset = W.qs; *bytes = (size_t)s.L * W.Mp * s.d * 2; break;
    case 10: *offset = W.os; *bytes = (size_t)s.L * W.Mp * s.d * 2; break;
    case 11: *offset = W.hs; *bytes = (size_t)s.L * W.Mp * s.Fp * 2; break;
    case 12: *offset = W.xgs; *bytes = (size_t)(2 * s.L + 1) * W.Mp * s.d * 2; break;
    case 13: *offset = W.zero; *bytes = kZeroBytes; break;
    default: return LLMCAD_EARG;
  }
  return LLMCAD_OK;
}

}  // extern "C"
