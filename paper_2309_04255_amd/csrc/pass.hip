// The whole verification pass (§3.2 of arXiv 2309.04255) as one persistent
// launch.
//
// Why one launch: a pass is a chain of five dependent steps per layer, each
// streaming tens to hundreds of MB of weights.  As separate kernels every
// step pays a ramp-up and a drain; here every workgroup (one per CU, all
// resident: cooperative launch) walks the phases in order and meets the
// others at a grid barrier between phases.  Weights never depend on the
// previous phase, so each workgroup issues the first weight loads of its
// next tile before it waits at the barrier, and HBM keeps streaming
// meanwhile.
//
// Phases: embed + tree prep; per layer QKV projection (RMSNorm scale,
// rotary embedding and K/V cache write in the epilogue) -> tree attention
// (ancestor mask) -> O projection (+residual) -> gate/up (RMSNorm scale;
// SwiGLU epilogue) -> down projection (+residual); then the final RMSNorm,
// the LM head + argmax, and the accept walk in the workgroup that completes
// the argmax.
//
// GEMM phases (activations X [Mp rows x K], packed weights W [N x K]): the
// 16-column blocks of a step are dealt out in contiguous runs, one run per
// workgroup, and every block is computed over the full K by one workgroup,
// so no partial sum leaves the CU and the epilogue follows the main loop
// directly (except the split-K projections of 64+ row passes, below).  The
// four waves take interleaved 32-wide k-steps; per k-step a wave loads one
// 1 KiB weight fragment per block (non-temporal: weights are read once) and
// one 1 KiB activation fragment per 16-row block -- the activations are
// stored in MFMA fragment order by the phase that produces them, so that
// read is one contiguous 1 KiB load that every CU of an XCD shares through
// L2.  The first weight stages go to LDS by direct global->LDS loads before
// the barrier; after it, both streams run through one register pipeline.
// The waves' partial tiles meet in LDS and are added in wave order
// (bit-reproducible).  Inputs of the epilogue that do not depend on the tile
// (the residual stream, rotary table, norm gains) are parked in LDS before
// the barrier.  Passes of 64+ rows add row-split tiles (the waves split the
// rows and share each weight fragment through LDS) and split-K groups for
// the projections with one block per workgroup; 4-bit weights have tiles of
// their own (codes dequantised on the matrix cores).
//
// Coherence without cache maintenance: every buffer handed from one phase to
// the next is written once per pass at its own address with device-coherent
// stores and read after the barrier with ordinary loads, so no L2 can hold an
// older copy; buffers reused within a pass (attention partials) are read
// with device-coherent loads.  Barriers and per-head joins are counters
// polled with bounded spins: a wait that exceeds its bound records an error
// status and the workgroup leaves the pass, so no wave can hang.
#include <math.h>

#include "device.h"
#include "kernels.h"
#include "layout.h"

namespace llmcad {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;

// Tuning constants of the GEMM phases (the defaults were measured best on the
// LLaMA-7B workload; -D overrides them for sweeps): the VGPRs (in units of 4)
// a tile's register pipeline may hold, its depth for one-block and for wider
// tiles, and the widest tile (in 16-column blocks) at 128 and at 64 rows (at
// 16 and 32 rows: 8, or 9 for a gate/up step marked wide).
#ifndef LLMCAD_STAGE_REGS
#define LLMCAD_STAGE_REGS 40
#endif
#ifndef LLMCAD_DEPTH_ONE
#define LLMCAD_DEPTH_ONE 8
#endif
#ifndef LLMCAD_DEPTH_WIDE
#define LLMCAD_DEPTH_WIDE 4
#endif
#ifndef LLMCAD_TILE_BLOCKS_MB8
#define LLMCAD_TILE_BLOCKS_MB8 4
#endif
#ifndef LLMCAD_TILE_BLOCKS_MB4
#define LLMCAD_TILE_BLOCKS_MB4 6
#endif

enum Epilogue { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_LOGITS = 3 };

// The launch parameters, read in place from the kernel-argument segment
// (constant memory): loads through a wave-uniform address of it are scalar
// loads, their values are wave-uniform, and no store can alias them.
typedef const LLMCAD_CONSTANT PassParams KParams;

// Inside a non-inlined function the compiler no longer knows that the
// parameter block's address is the same in every lane; re-establish it.
__device__ __forceinline__ KParams& uniform_params(KParams& p) {
  const uint64_t v = (uint64_t)&p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return *(KParams*)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ bf16x8 ldg_nt(const bf16x8* p) {
  return __builtin_nontemporal_load((const LLMCAD_GLOBAL bf16x8*)p);
}

// The pointer as a value the compiler cannot see through: a load from a
// pointer chosen by a condition stays one unconditional load (the compiler
// would otherwise turn the choice into a branch around the load, and a load
// that may or may not have been issued makes every later wait a full drain).
template <class T>
__device__ __forceinline__ const T* opaque(const T* p) {
  asm volatile("" : "+v"(p));
  return p;
}

// Element offset of (row, col) in a fragment-order bf16 [Mp][K] matrix with
// MB 16-row blocks: block (col / 32, row / 16) is 1 KiB at
// ((col / 32) MB + row / 16) KiB, and holds row 16 rb + l % 16, columns
// 32 s + 8 (l / 16) + e at lane l, element e -- the A operand of one
// 16x16x32 MFMA.
__device__ __forceinline__ size_t frag_off(int row, int col, int MB) {
  return ((size_t)((col >> 5) * MB + (row >> 4)) * 64 + (row & 15) + 16 * ((col >> 3) & 3)) * 8 +
         (col & 7);
}

// Workgroups are dispatched to the GPU's 8 XCDs round-robin (workgroup w
// runs on XCD w % 8).  Phases deal out their work by this virtual index,
// which runs XCD by XCD: each XCD gets a contiguous, equal share, so shares
// that differ by a block spread evenly over the XCDs (dealt by w itself,
// every 8th workgroup would take the larger share, all on the same XCDs).
constexpr int kXcds = 8;
__device__ __forceinline__ int virtual_wg(int G) {
  const int w = blockIdx.x;
  return G % kXcds == 0 ? (w % kXcds) * (G / kXcds) + w / kXcds : w;
}

// ------------------------------------------------------------------ sync

struct Sync {
  int* bar;
  int* status;
  int limit;
  int* lds_flag;
  long long* trace;  // [phase][8] timestamps of this workgroup, or null
};

__device__ __forceinline__ Sync make_sync(KParams& p, int* lds_flag) {
  Sync s;
  s.bar = p.bar;
  s.status = p.status;
  s.limit = p.spin_limit;
  s.lds_flag = lds_flag;
  s.trace = p.trace != nullptr ? p.trace + (size_t)blockIdx.x * pass_phases(p.L) * 8 : nullptr;
  return s;
}

// Diagnostics: wall-clock (100 MHz) marks per phase: 0 = barrier wait
// entered, 1 = wait over, 2 = phase work done; GEMM phases also mark 3 =
// activation stream started, 4 = first tile's main loop done, 5 = all tiles
// and epilogues done (in the LM head's walking workgroup 6 = walk started,
// 7 = walk done); the attention marks 3 = loads issued, 4 = keys done,
// 5 = result stored, and in a merging split 6 = the other splits' arrivals
// seen, 7 = their partials loaded.
__device__ __forceinline__ void trace_mark(const Sync& s, int phase, int k) {
  if (s.trace != nullptr && threadIdx.x == 0) stg(s.trace + phase * 8 + k, (long long)wall_clock64());
}

// End of a phase: this workgroup's stores have completed, then one
// device-scope increment on its barrier counter (workgroup g counts on
// counter g % kBarSlots, so arrivals do not serialise on one address).
__device__ __forceinline__ void grid_arrive(const Sync& s, int phase) {
  trace_mark(s, phase, 2);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) atomic_add_dev(s.bar + (blockIdx.x % kBarSlots) * kBarStride, 1);
}

// Polled by one wave: returns 1 once all G workgroups have arrived `phase`
// times (every lane reads one counter), 0 if the bounded spin ran out (the
// pass status is then set).  The total is exact only because every
// workgroup waits at every phase before it arrives again: no workgroup can
// then be more than one arrival ahead.
__device__ __forceinline__ int poll_grid(const Sync& s, int phase, int G) {
  const int lane = threadIdx.x & 63;
  const int slots = G < kBarSlots ? G : kBarSlots;
  const int per = G / kBarSlots + (lane < G % kBarSlots ? 1 : 0);
  const int want = lane < slots ? phase * (G < kBarSlots ? 1 : per) : 0;
  const int* slot = s.bar + (lane < slots ? lane : 0) * kBarStride;
  if (s.limit < 0) {  // (diagnostics: every grid wait gives up at once)
    if (lane == 0) st_coherent(s.status, 1);
    return 0;
  }
  int spins = 0;
  while (true) {
    const int v = lane < slots ? ld_coherent(slot) : 0;
    if (__all(v >= want)) return 1;
    __builtin_amdgcn_s_sleep(1);
    if (++spins > s.limit) {
      if (lane == 0) st_coherent(s.status, 1);
      return 0;
    }
  }
}

// Waits until all G workgroups have arrived `phase` times; wave 0 polls.
// False (to all threads) if the bounded spin ran out.
__device__ __forceinline__ bool grid_wait(const Sync& s, int phase, int G) {
  if (threadIdx.x < 64) {
    const int ok = poll_grid(s, phase, G);
    if (threadIdx.x == 0) *s.lds_flag = ok;
  }
  // (LDS-only barriers: the other waves may have weight loads in flight,
  // which must not be drained here)
  lds_barrier();
  const bool ok = *s.lds_flag != 0;
  lds_barrier();
  return ok;
}

// ------------------------------------------------------------------ GEMM

struct GemmLds {
  // (the LM head needs no RMSNorm scales: it reuses their room for its
  // softmax normalisers)
  union {
    float rstd[kMaxNodes];      // RMSNorm scale per row
    float best_s[kMaxNodes];    // LM head: sum of exp(logit - best_v) per row over this workgroup's blocks
  };
  union {
    float part_ss[1024];        // its partial sums
    float red_s[kMaxNodes][8];  // LM head: sum of exp(logit - red_v) per (row, block of the tile)
  };
  float red_v[kMaxNodes][8];    // LM head: argmax per (row, block of the tile)
  int red_i[kMaxNodes][8];
  float best_v[kMaxNodes];      // LM head: argmax per row over this workgroup's blocks
  int best_i[kMaxNodes];
  int reach[kMaxNodes];         // accept walk: reachability of each node,
  int jump[kMaxNodes];          // its pointer-jumping ancestor, then the path by depth
  int amax[kMaxNodes];
  int tok[kMaxNodes];  // accept walk: the tree, staged from the workspace
  int par[kMaxNodes];
  int dep[kMaxNodes];
  int walk_len;
};

// LDS of a GEMM tile of cw blocks (dynamic shared memory), in KiB, with
// SL partial-tile slots:
//   [0, SL cw MB)                the partial tiles, fp32 [SL][cw][MB][64 lanes][4]:
//                                the four waves' (SL = 4), or two sums of
//                                two waves' (SL = 2, when four slots and the
//                                epilogue inputs would not fit), or a split-K
//                                group's partial sums (SL = S)
//   [SL cw MB, (SL+1) cw MB + cw)  epilogue inputs: per (block, row block) 1 KiB
//                                of the residual stream (fp32 [16 rows][16]) or
//                                of the rotary table (fp32 [16 rows][8 pairs][2]);
//                                then per block 1 KiB holding its 16 norm gains
//                                (bf16, first 32 bytes)
//   [(SL+1) cw MB + cw, 142)     the first weight stages of each wave, copied
//                                before the phase's barrier
constexpr int kGemmLdsBytes = 142 * 1024;
__host__ __device__ constexpr int tw_off() { return 0; }
__host__ __device__ constexpr int epi_off(int cw, int MB, int SL) { return SL * cw * MB * 1024; }
__host__ __device__ constexpr int wl_off(int cw, int MB, int SL) { return ((SL + 1) * cw * MB + cw) * 1024; }
// partial-tile slots of a tile: four, or two (or one) when four (two) do not fit
__host__ __device__ constexpr int tile_slots(int cw, int MB) {
  return wl_off(cw, MB, 4) <= kGemmLdsBytes ? 4 : wl_off(cw, MB, 2) <= kGemmLdsBytes ? 2 : 1;
}

// Direct global -> LDS copy of 16 bytes per lane: lane l's bytes land at
// lds + 16 l.  `lds` must be the same in every lane.
__device__ __forceinline__ void dma16(const void* src, char* lds) {
  __builtin_amdgcn_global_load_lds((const LLMCAD_GLOBAL void*)src,
                                   (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}

// Where the epilogue of one GEMM step writes in a given layer, and the sums
// of squares of the residual version a norm step reads.  Every field is
// assigned for every step by branch-free selects: built behind a switch on
// the (run-time) step, the structure would live in scratch memory, and each
// output store would first wait for a scratch reload queued behind the
// previous store.
struct StepIo {
  const float* ssq;  // norm steps: [d/16][Mp] sums of squares of the residual version
  bf16* q;           // QKV: [Mp][d] queries after the rotary embedding
  bf16* kc;          // QKV: K cache of this layer [H][cap][Dh]
  bf16* vc;          // QKV: V cache of this layer, transposed per head [H][Dh][cap]
  float* x_out;      // RESID: [Mp][d]
  float* ssq_out;    // RESID: [d/16][Mp]
  bf16* xg_out;      // RESID: fragment-order bf16(x_out * g_next)
  bf16* h;           // SWIGLU: fragment-order [Mp][Fp]
};

template <int EPI>
__device__ __forceinline__ StepIo step_io(KParams& p, int step, int l) {
  const size_t xsz = (size_t)p.Mp * p.d, ssz = (size_t)p.d_nb * p.Mp;
  const size_t kv = (size_t)l * p.H * p.cap * p.Dh;
  // residual version read by a norm step (QKV 2l, gate/up 2l+1) or written
  // by a residual step (O 2l+1, down 2l+2)
  const int ver_in = EPI == EPI_SWIGLU ? 2 * l + 1 : 2 * l;
  const int ver_out = step == STEP_DOWN ? 2 * l + 2 : 2 * l + 1;
  StepIo io;
  io.ssq = p.ssq + (size_t)ver_in * ssz;
  io.q = p.q + (size_t)l * xsz;
  io.kc = p.k_cache + kv;
  io.vc = p.v_cache + kv;
  io.x_out = p.x + (size_t)ver_out * xsz;
  io.ssq_out = p.ssq + (size_t)ver_out * ssz;
  io.xg_out = p.xg + (size_t)ver_out * xsz;
  io.h = p.h + (size_t)l * p.Mp * p.Fp;
  return io;
}

// What a tile's main loop reads, with every field assigned for every step
// (branch-free selects: the compiler keeps this in registers).
struct TileIn {
  const bf16x8* w;     // packed matrix (4-bit: its codes)
  const uint16_t* sc;  // 4-bit: its packed scales (bf16 bits)
  const bf16x8* a;     // fragment-order activations
  const float* ssq;    // norm steps: [d/16][Mp] sums of squares; else null
  const float* x_in;   // residual steps: [Mp][d]; else null
  const bf16* g_next;  // residual steps: gain of the next norm; else null
  int ks;
  bool norm, resid;
};

__device__ __forceinline__ TileIn tile_in(KParams& p, int step, int l) {
  const size_t xsz = (size_t)p.Mp * p.d, ssz = (size_t)p.d_nb * p.Mp;
  const char* lw = p.packed + p.layer0 + (long long)l * p.layer_bytes;
  const StepPlan& sp = p.step[step];
  TileIn t;
  t.w = (const bf16x8*)((sp.layer_rel ? lw : p.packed) + sp.w_off);
  t.sc = (const uint16_t*)((sp.layer_rel ? lw : p.packed) + sp.s_off);
  t.ks = sp.ksteps;
  t.resid = step == STEP_O || step == STEP_DOWN;
  t.norm = step == STEP_QKV || step == STEP_GATE_UP;
  // x version read by a norm step: QKV 2l, GU 2l+1, LM 2L; residual input: O 2l, DOWN 2l+1
  const int ver = step == STEP_LM ? 2 * p.L : (step == STEP_GATE_UP || step == STEP_DOWN) ? 2 * l + 1 : 2 * l;
  const bf16* act = step == STEP_O ? p.o + (size_t)l * xsz
                  : step == STEP_DOWN ? p.h + (size_t)l * p.Mp * p.Fp
                  : step == STEP_LM ? p.xnf
                                      : p.xg + (size_t)ver * xsz;
  t.a = (const bf16x8*)act;
  t.ssq = t.norm ? p.ssq + (size_t)ver * ssz : nullptr;
  t.x_in = t.resid ? p.x + (size_t)ver * xsz : nullptr;
  const bf16* g_o = (const bf16*)(lw + p.o_ffn_norm);
  const bf16* g_d = l + 1 < p.L ? (const bf16*)(lw + p.layer_bytes + p.o_attn_norm)
                                : (const bf16*)(p.packed + p.o_final_norm);
  t.g_next = step == STEP_O ? g_o : step == STEP_DOWN ? g_d : nullptr;
  return t;
}

// Register stages per wave: at most ~160 VGPRs of them, and few -- 8 for
// one-block tiles, 4 for wider ones.  The bytes in flight across a barrier
// come mostly from the stages copied to LDS before it; a deeper register
// pipeline only lengthens the queues in the memory system (on the 7B
// workload 8 and 4 stages beat the 13, 8 and 5 that fill ~160 VGPRs by
// 3%), and a depth that divides the LDS stages lets the copy use them all.
template <int MB, int C>
constexpr int tile_depth() {
  constexpr int regs = LLMCAD_STAGE_REGS / (C + MB);
  constexpr int cap = C == 1 ? LLMCAD_DEPTH_ONE : LLMCAD_DEPTH_WIDE;
  constexpr int d = regs < cap ? regs : cap;
  return d < 2 ? 2 : d;
}

// One tile: blocks [nb0, nb0 + C) of a step over all its k-steps.  Issues
// the first weight stages, then (wait_phase >= 0) waits at the grid barrier
// for the step's inputs, starts the activation stream and the epilogue
// inputs, streams both through the MFMAs and leaves the waves' partial tiles
// in LDS.  False if a wait ran out.
template <int MB, int C>
__device__ __attribute__((noinline, not_tail_called)) bool tile_compute(KParams& pin, int step, int layer,
                                                                       int nb0, int wait_phase, char* lds,
                                                                       GemmLds& gl, int* lds_flag, int k0,
                                                                       int kn, int epi_in) {
  KParams& p = uniform_params(pin);
  step = wave_uniform(step);
  layer = wave_uniform(layer);
  nb0 = wave_uniform(nb0);
  wait_phase = wave_uniform(wait_phase);
  k0 = wave_uniform(k0);
  epi_in = wave_uniform(epi_in);
  const TileIn io = tile_in(p, step, layer);
  const int wave = wave_index(), lane = threadIdx.x & 63;
  // k-steps [k0, k0 + kn) of the step's io.ks (a split-K slice; all of them otherwise)
  const int ks = wave_uniform(kn);
  const int ns = wave_uniform(wave < ks ? (ks - wave + kWaves - 1) / kWaves : 0);
  // Pipeline depth (tile_depth), but no deeper than the LDS stages that
  // fit, so that wide tiles still get some (the LDS phase advances D stages
  // at a time).
  constexpr int SL = tile_slots(C, MB);
  constexpr int WL_STAGES = (kGemmLdsBytes - wl_off(C, MB, SL)) / (kWaves * C * 1024);
  constexpr int D0 = tile_depth<MB, C>();
  constexpr int D = WL_STAGES >= 2 && WL_STAGES < D0 ? WL_STAGES : D0;
  // this wave's k-steps: k0 + wave + 4 i
  const bf16x8* wt = io.w + ((size_t)nb0 * io.ks + k0 + wave) * 64 + lane;
  const size_t cstride = (size_t)io.ks * 64;
  const bf16x8* at = io.a + (size_t)(k0 + wave) * MB * 64 + lane;
  // Loads past the wave's last k-step read a line of zeros instead (the
  // load is still issued, so that the compiler's count of loads in flight
  // stays exact and every wait in the loop is for one stage only).  For the
  // same reason every load of a tile is unconditional: inputs a step does
  // not have are read from the zero line too.
  const bf16x8* zero = (const bf16x8*)p.zero + lane;
  const f32x4* zero4 = (const f32x4*)p.zero + lane;
  bf16x8 bw[D][C];
  bf16x8 ba[D][MB];
  // The first P stages of the wave's weights are copied into LDS before the
  // barrier (P a multiple of D, as many as fit); the register pipeline
  // starts at stage P.
  constexpr int PMAX = WL_STAGES / D * D;
  const int wcap = wave_uniform(p.step[step].wl_cap);
  const int pcap = wave_uniform(wcap < PMAX ? wcap / D * D : PMAX);
  const int P = wave_uniform(wait_phase >= 0 ? (ns / D * D < pcap ? ns / D * D : pcap) : 0);
  char* wl = lds + wl_off(C, MB, SL) + (size_t)wave * PMAX * C * 1024;
  auto load_w = [&](int slot, int i, bool want) {  // stage i, or nothing (zero line)
    const bool live = want && i < ns;
#pragma unroll
    for (int c = 0; c < C; ++c) bw[slot][c] = ldg_nt(opaque(live ? wt + c * cstride + (size_t)(kWaves * i) * 64 : zero));
  };
  auto load_a = [&](int slot, int i) {
    const bool live = i < ns;
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) ba[slot][rb] = ldg(opaque(live ? at + ((size_t)kWaves * i * MB + rb) * 64 : zero));
  };

  // Before the barrier, waves 1-3 start the weight stream: each its own
  // LDS stages (wave 1 also wave 0's), then its register stages.  Wave 0
  // polls the barrier and issues no load before it has seen it (a poll
  // waits for every older load of its wave).
  const int ns0 = (ks + kWaves - 1) / kWaves;
  const int P0 = wave_uniform(wait_phase >= 0 ? (ns0 / D * D < pcap ? ns0 / D * D : pcap) : 0);
  // Epilogue inputs (residual stream or rotary table, and the next norm's
  // gains; written two or more phases ago, so they need no barrier), by the
  // last wave before the barrier: per (block, row block) unit 16 B per lane,
  // then each block's gains, parked in LDS once they land -- before that
  // wave's weight stages, so that the wait is for them alone (a wait behind
  // a direct-to-LDS loop is a full drain).  After the barrier only the
  // activations are then on the critical path.
  constexpr int KU = C * MB;
  constexpr int kEpiWave = kWaves - 1;
  f32x4 sx[KU], sg[C];
  if (wave == kEpiWave && epi_in) {
    const bool resid = io.resid;
#pragma unroll
    for (int u = 0; u < KU; ++u) {
      const int c = u / MB, rb = u % MB;
      const int col0 = kNB * (nb0 + c);
      const f32x4* src = zero4;
      if (resid) {  // residual rows 16 rb + l / 4, columns col0 + 4 (l % 4) .. + 3
        src = (const f32x4*)(io.x_in + (size_t)(16 * rb + (lane >> 2)) * p.d + col0 + 4 * (lane & 3));
      } else if (step == STEP_QKV && col0 < 2 * p.d) {  // (cos, sin) of pairs 8 t + 2 (l % 4), + 1
        const int t = (col0 % p.d % p.Dh) / kNB;
        src = (const f32x4*)(p.rope + ((size_t)(16 * rb + (lane >> 2)) * (p.Dh / 2) + 8 * t + 2 * (lane & 3)) * 2);
      }
      sx[u] = ldg(opaque(src));
    }
#pragma unroll
    for (int c = 0; c < C; ++c)
      sg[c] = ldg(opaque(resid ? (const f32x4*)(io.g_next + kNB * (nb0 + c) + 8 * (lane & 1)) : zero4));
#pragma unroll
    for (int u = 0; u < KU; ++u) lds_st<f32x4>(lds + epi_off(C, MB, SL) + (size_t)u * 1024 + lane * 16, sx[u]);
#pragma unroll
    for (int c = 0; c < C; ++c) lds_st<f32x4>(lds + epi_off(C, MB, SL) + (size_t)(C * MB + c) * 1024 + lane * 16, sg[c]);
  }
  if (wave != 0) {
    if constexpr (PMAX > 0) {
      for (int i = 0; i < P; ++i)
#pragma unroll
        for (int c = 0; c < C; ++c)
          dma16(wt + c * cstride + (size_t)(kWaves * i) * 64, wl + (size_t)(i * C + c) * 1024);
      if (wave == 1) {
        const bf16x8* wt0 = wt - 64;
        char* wl0 = lds + wl_off(C, MB, SL);
        for (int i = 0; i < P0; ++i)
#pragma unroll
          for (int c = 0; c < C; ++c)
            dma16(wt0 + c * cstride + (size_t)(kWaves * i) * 64, wl0 + (size_t)(i * C + c) * 1024);
      }
    }
#pragma unroll
    for (int u = 0; u < D; ++u) load_w(u, P + u, true);
  }
  __builtin_amdgcn_sched_barrier(0);
  if (wait_phase >= 0) {
    const Sync sy = make_sync(p, lds_flag);
    trace_mark(sy, wait_phase, 0);
    if (!grid_wait(sy, wait_phase, p.G)) return false;
    trace_mark(sy, wait_phase, 1);
  }
  // A norm step's sums of squares (written by the previous phase), held in
  // registers through the main loop: thread t takes rows 4 q .. 4 q + 3
  // (q = t % (Mp / 4)) of the 16-column blocks of chunk t / (Mp / 4).
  constexpr bool SSQR = MB <= 2;
  constexpr int SSQN = SSQR ? 8 : 1;
  f32x4 sr[SSQN];
  if constexpr (SSQR) {
    constexpr int QUADS = 4 * MB, CH = 256 / QUADS;
    const int q = threadIdx.x % QUADS, ch = threadIdx.x / QUADS;
    const int t0 = ch * p.d_nb / CH, t1 = (ch + 1) * p.d_nb / CH;
    const bool on = io.norm && p.ssq_regs;
#pragma unroll
    for (int k = 0; k < SSQN; ++k)
      sr[k] = ldg(opaque(on && t0 + k < t1 ? (const f32x4*)(io.ssq + (size_t)(t0 + k) * (16 * MB) + 4 * q) : zero4));
  }
#pragma unroll
  for (int u = 0; u < D; ++u) load_a(u, u);
  // Every load so far has landed (the direct-to-LDS copies among them; from
  // here on only register loads are in flight, so that the loop's waits can
  // count them exactly), and wave 0's LDS stages, copied by wave 1, are
  // visible to it.  Then wave 0's register stages.
  __builtin_amdgcn_s_waitcnt(0);
  lds_barrier();
  if (wave == 0) {
#pragma unroll
    for (int u = 0; u < D; ++u) load_w(u, P + u, true);
  }
  __builtin_amdgcn_sched_barrier(0);
  if (wait_phase >= 0 && p.trace != nullptr && threadIdx.x == 0)
    stg(p.trace + (size_t)blockIdx.x * pass_phases(p.L) * 8 + wait_phase * 8 + 3, (long long)wall_clock64());

  f32x4 acc[MB][C];
#pragma unroll
  for (int rb = 0; rb < MB; ++rb)
#pragma unroll
    for (int c = 0; c < C; ++c) acc[rb][c] = f32x4{0.f, 0.f, 0.f, 0.f};
  // Stages [0, P) from LDS (only activation loads in flight), then the
  // register pipeline, whose first D stages came with the prologue.  (Steps
  // past the end multiply zero lines: no guard, so the loops are
  // straight-line code and every wait covers one stage.)
  int i = 0;
  for (; i < P; i += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      __builtin_amdgcn_sched_barrier(0);
      bf16x8 b[C];
#pragma unroll
      for (int c = 0; c < C; ++c) b[c] = lds_ld<bf16x8>(wl + (size_t)((i + u) * C + c) * 1024 + lane * 16);
#pragma unroll
      for (int rb = 0; rb < MB; ++rb)
#pragma unroll
        for (int c = 0; c < C; ++c) acc[rb][c] = mfma16x16x32(ba[u][rb], b[c], acc[rb][c]);
      __builtin_amdgcn_sched_barrier(0);
      load_a(u, i + u + D);
    }
  }
  for (; i + D < ns; i += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int rb = 0; rb < MB; ++rb)
#pragma unroll
        for (int c = 0; c < C; ++c) acc[rb][c] = mfma16x16x32(ba[u][rb], bw[u][c], acc[rb][c]);
      __builtin_amdgcn_sched_barrier(0);
      load_w(u, i + u + D, true);
      load_a(u, i + u + D);
    }
  }
  // the last round: nothing left to load (no zero-line loads for the
  // barrier at the end of the tile to wait for)
  if (i < ns) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int rb = 0; rb < MB; ++rb)
#pragma unroll
        for (int c = 0; c < C; ++c) acc[rb][c] = mfma16x16x32(ba[u][rb], bw[u][c], acc[rb][c]);
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (SSQR) {
    if (io.norm && p.ssq_regs) {
      constexpr int QUADS = 4 * MB;
      const int q = threadIdx.x % QUADS, ch = threadIdx.x / QUADS;
      f32x4 t = sr[0];
#pragma unroll
      for (int k = 1; k < SSQN; ++k) t += sr[k];
      *(f32x4*)&gl.part_ss[ch * 16 * MB + 4 * q] = t;
    }
  }
  // This wave's partial tile -> LDS; the epilogue adds the four in wave
  // order.  With two slots, waves 2 and 3 hand theirs to waves 0 and 1
  // first, and the epilogue adds (w0 + w2) + (w1 + w3); with one, the waves
  // add theirs into it in turn: ((w3 + w2) + w1) + w0.
  if constexpr (SL == 1) {
#pragma unroll 1
    for (int w = kWaves - 1; w >= 0; --w) {
      if (wave == w) {
#pragma unroll
        for (int c = 0; c < C; ++c)
#pragma unroll
          for (int rb = 0; rb < MB; ++rb) {
            char* at1 = lds + tw_off() + ((size_t)(c * MB + rb) * 64 + lane) * 16;
            lds_st<f32x4>(at1, w == kWaves - 1 ? acc[rb][c] : lds_ld<f32x4>(at1) + acc[rb][c]);
          }
      }
      __syncthreads();
    }
  } else if constexpr (SL == 2) {
    if (wave >= 2) {
#pragma unroll
      for (int c = 0; c < C; ++c)
#pragma unroll
        for (int rb = 0; rb < MB; ++rb)
          lds_st<f32x4>(lds + tw_off() + ((size_t)(((wave - 2) * C + c) * MB + rb) * 64 + lane) * 16, acc[rb][c]);
    }
    __syncthreads();
    if (wave < 2) {
#pragma unroll
      for (int c = 0; c < C; ++c)
#pragma unroll
        for (int rb = 0; rb < MB; ++rb) {
          char* at2 = lds + tw_off() + ((size_t)((wave * C + c) * MB + rb) * 64 + lane) * 16;
          lds_st<f32x4>(at2, acc[rb][c] + lds_ld<f32x4>(at2));
        }
    }
  } else {
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
      for (int rb = 0; rb < MB; ++rb)
        lds_st<f32x4>(lds + tw_off() + ((size_t)((wave * C + c) * MB + rb) * 64 + lane) * 16, acc[rb][c]);
  }
  __syncthreads();
  return true;
}

// ---- row-split tiles (passes of 64 or more rows)
//
// A K-split tile keeps every wave's accumulators for all MB row blocks, which
// caps it at a few blocks at 64 and 128 rows, so a workgroup with more blocks
// than that reads the whole activation matrix once per tile.  Here the waves
// split the rows instead: wave w owns row blocks [w MB/4, (w + 1) MB/4) of
// every k-step of the tile's C blocks, so a tile takes up to 8 blocks and its
// workgroup reads the activations once.  Per k-step wave w loads the weight
// fragments of blocks w, w + 4 (a quarter of the tile) and its own row
// blocks' activation fragments through its register pipeline, writes its
// weight fragments to one of two LDS buffers, and after the workgroup's
// barrier reads all C of them from there.  No partial sums cross waves: each
// wave writes its rows' tiles to the one partial-tile slot.
template <int MB, int C>
__device__ __attribute__((noinline, not_tail_called)) bool tile_compute_rows(KParams& pin, int step, int layer,
                                                                            int nb0, int wait_phase, char* lds,
                                                                            int* lds_flag) {
  KParams& p = uniform_params(pin);
  step = wave_uniform(step);
  layer = wave_uniform(layer);
  nb0 = wave_uniform(nb0);
  wait_phase = wave_uniform(wait_phase);
  const TileIn io = tile_in(p, step, layer);
  const int wave = wave_index(), lane = threadIdx.x & 63;
  constexpr int RB = MB / kWaves;              // row blocks per wave
  constexpr int NW = (C + kWaves - 1) / kWaves;  // weight fragments per wave per k-step
  static_assert(RB >= 1 && RB * kWaves == MB, "row-split tiles need 4 or 8 row blocks");
  constexpr int DR = LLMCAD_STAGE_REGS / (NW + RB);
  constexpr int D = DR < 2 ? 2 : DR > 8 ? 8 : DR;
  const int ks = wave_uniform(io.ks);
  const size_t cstride = (size_t)ks * 64;
  const bf16x8* at = io.a + (size_t)(wave * RB) * 64 + lane;
  const bf16x8* zero = (const bf16x8*)p.zero + lane;
  const f32x4* zero4 = (const f32x4*)p.zero + lane;
  bf16x8 bw[D][NW];
  bf16x8 ba[D][RB];
  // this wave's weight fragments: blocks wave + 4 j (j < NW) of the tile
  auto load_w = [&](int slot, int i) {  // k-step i, or the zero line past the last
#pragma unroll
    for (int j = 0; j < NW; ++j) {
      const int c = wave + kWaves * j;
      const bool live = i < ks && c < C;
      bw[slot][j] = ldg_nt(opaque(live ? io.w + ((size_t)(nb0 + c) * ks + i) * 64 + lane : zero));
    }
  };
  auto load_a = [&](int slot, int i) {
    const bool live = i < ks;
#pragma unroll
    for (int r = 0; r < RB; ++r) ba[slot][r] = ldg(opaque(live ? at + ((size_t)i * MB + r) * 64 : zero));
  };
  char* wbuf = lds;  // two buffers of C KiB: k-step i's fragments in buffer i % 2, block c at c KiB
  // Waves 1-3 start their weight stages before the barrier; wave 0 polls it
  // with no load in flight (a poll waits for every older load of its wave).
  if (wave != 0) {
#pragma unroll
    for (int u = 0; u < D; ++u) load_w(u, u);
  }
  __builtin_amdgcn_sched_barrier(0);
  if (wait_phase >= 0) {
    const Sync sy = make_sync(p, lds_flag);
    trace_mark(sy, wait_phase, 0);
    if (!grid_wait(sy, wait_phase, p.G)) return false;
    trace_mark(sy, wait_phase, 1);
  }
  if (wave == 0) {
#pragma unroll
    for (int u = 0; u < D; ++u) load_w(u, u);
  }
#pragma unroll
  for (int u = 0; u < D; ++u) load_a(u, u);
  __builtin_amdgcn_sched_barrier(0);
  if (wait_phase >= 0 && p.trace != nullptr && threadIdx.x == 0)
    stg(p.trace + (size_t)blockIdx.x * pass_phases(p.L) * 8 + wait_phase * 8 + 3, (long long)wall_clock64());
  f32x4 acc[RB][C];
#pragma unroll
  for (int r = 0; r < RB; ++r)
#pragma unroll
    for (int c = 0; c < C; ++c) acc[r][c] = f32x4{0.f, 0.f, 0.f, 0.f};
  // one k-step from register stage u: share the weights, multiply, refill
  auto kstep = [&](int i, int u, bool refill) {
    char* buf = wbuf + (size_t)(i & 1) * C * 1024;
#pragma unroll
    for (int j = 0; j < NW; ++j) {
      const int c = wave + kWaves * j;
      if (c < C) lds_st<bf16x8>(buf + (size_t)c * 1024 + lane * 16, bw[u][j]);
    }
    lds_barrier();  // (the other buffer's readers are past the previous barrier)
#pragma unroll
    for (int c = 0; c < C; ++c) {
      const bf16x8 b = lds_ld<bf16x8>(buf + (size_t)c * 1024 + lane * 16);
#pragma unroll
      for (int r = 0; r < RB; ++r) acc[r][c] = mfma16x16x32(ba[u][r], b, acc[r][c]);
    }
    if (refill) {
      load_w(u, i + D);
      load_a(u, i + D);
    }
  };
  int i = 0;
  for (; i + D < ks; i += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) kstep(i + u, u, true);
  }
#pragma unroll
  for (int u = 0; u < D; ++u)
    if (i + u < ks) kstep(i + u, u, false);
  lds_barrier();  // (every wave is done with the weight buffers)
  // this wave's rows -> the one slot: unit (block c, row block rb) at (c MB + rb) KiB
#pragma unroll
  for (int c = 0; c < C; ++c)
#pragma unroll
    for (int r = 0; r < RB; ++r)
      lds_st<f32x4>(lds + tw_off() + ((size_t)(c * MB + wave * RB + r) * 64 + lane) * 16, acc[r][c]);
  // epilogue inputs (written two or more phases ago): per (block, row block)
  // the residual rows or the rotary table, then each block's gains
  char* epi = lds + epi_off(C, MB, 1);
  const bool resid = io.resid;
  for (int u = wave; u < C * MB; u += kWaves) {
    const int c = u / MB, rb = u % MB;
    const int col0 = kNB * (nb0 + c);
    const f32x4* src = zero4;
    if (resid) {
      src = (const f32x4*)(io.x_in + (size_t)(16 * rb + (lane >> 2)) * p.d + col0 + 4 * (lane & 3));
    } else if (step == STEP_QKV && col0 < 2 * p.d) {
      const int t = (col0 % p.d % p.Dh) / kNB;
      src = (const f32x4*)(p.rope + ((size_t)(16 * rb + (lane >> 2)) * (p.Dh / 2) + 8 * t + 2 * (lane & 3)) * 2);
    }
    lds_st<f32x4>(epi + (size_t)u * 1024 + lane * 16, ldg(opaque(src)));
  }
  for (int c = wave; c < C; c += kWaves)
    lds_st<f32x4>(epi + (size_t)(C * MB + c) * 1024 + lane * 16,
                  ldg(opaque(resid ? (const f32x4*)(io.g_next + kNB * (nb0 + c) + 8 * (lane & 1)) : zero4)));
  __syncthreads();
  return true;
}

template <int MB, int C>
__device__ __forceinline__ bool tile_dispatch_rows(int cw, KParams& p, int step, int layer, int nb0,
                                                   int wait_phase, char* lds, int* flag) {
  if constexpr (C >= 1) {
    if (cw == C) return tile_compute_rows<MB, C>(p, step, layer, nb0, wait_phase, lds, flag);
    return tile_dispatch_rows<MB, C - 1>(cw, p, step, layer, nb0, wait_phase, lds, flag);
  } else {
    return false;
  }
}

// ---- 4-bit weights

// The B operand of one k-step from its dword of packed codes (see pack.hip):
// the bf16 values 128 + q_e, formed by placing each code in the low mantissa
// bits of 128 (exact: 128 + q < 256 has 8 significant bits).
__device__ __forceinline__ bf16x8 q4_operand(uint32_t w) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  u32x4 v;
#pragma unroll
  for (int p2 = 0; p2 < 4; ++p2) v[p2] = ((w >> (4 * p2)) & 0x000F000Fu) | 0x43004300u;
  return __builtin_bit_cast(bf16x8, v);
}

// 4-bit tile: blocks [nb0, nb0 + C) of a layer step over all its scale
// groups (128 inputs, four k-steps each), waves taking interleaved groups.
// Per group the codes enter the matrix cores as 128 + q, and a product with
// a constant operand of 136 = 128 + 8 gives 136 times the group's sum of
// activations per row; their difference is sum_k (q_k - 8) a_k exactly as
// fp32 sums, and the column's scale multiplies it into the accumulator --
// w = s (q - 8) is never formed.  Structure as tile_compute (weight stages
// before the barrier, epilogue inputs parked in LDS by the last wave, partial
// tiles to LDS at the end), with register stages only.
template <int MB, int C>
__device__ __attribute__((noinline, not_tail_called)) bool tile_compute_q4(KParams& pin, int step, int layer,
                                                                          int nb0, int wait_phase, char* lds,
                                                                          GemmLds& gl, int* lds_flag) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  KParams& p = uniform_params(pin);
  step = wave_uniform(step);
  layer = wave_uniform(layer);
  nb0 = wave_uniform(nb0);
  wait_phase = wave_uniform(wait_phase);
  const TileIn io = tile_in(p, step, layer);
  const int wave = wave_index(), lane = threadIdx.x & 63;
  const int gs = io.ks;  // scale groups
  const int ns = wave_uniform(wave < gs ? (gs - wave + kWaves - 1) / kWaves : 0);
  constexpr int D = 2;
  // this wave's groups: wave + 4 i
  const u32x4* wt = (const u32x4*)io.w + ((size_t)nb0 * gs + wave) * 64 + lane;
  const size_t cstride = (size_t)gs * 64;
  const uint16_t* st = io.sc + ((size_t)nb0 * gs + wave) * kNB + (lane & 15);
  const size_t sstride = (size_t)gs * kNB;
  const bf16x8* at = io.a + (size_t)wave * 4 * MB * 64 + lane;
  const u32x4* zero_w = (const u32x4*)p.zero + lane;
  const uint16_t* zero_s = (const uint16_t*)p.zero;
  const bf16x8* zero = (const bf16x8*)p.zero + lane;
  const f32x4* zero4 = (const f32x4*)p.zero + lane;
  u32x4 bw[D][C];
  uint32_t bs[D][C];
  bf16x8 ba[D][4][MB];
  auto load_w = [&](int slot, int i) {  // group i of this wave, or the zero line past the last
    const bool live = i < ns;
#pragma unroll
    for (int c = 0; c < C; ++c) {
      bw[slot][c] = __builtin_nontemporal_load(
          (const LLMCAD_GLOBAL u32x4*)opaque(live ? wt + c * cstride + (size_t)(kWaves * i) * 64 : zero_w));
      bs[slot][c] = ldg(opaque(live ? st + c * sstride + (size_t)(kWaves * i) * kNB : zero_s));
    }
  };
  auto load_a = [&](int slot, int i) {
    const bool live = i < ns;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int rb = 0; rb < MB; ++rb)
        ba[slot][t][rb] = ldg(opaque(live ? at + ((size_t)kWaves * 4 * i * MB + t * MB + rb) * 64 : zero));
  };
  // Epilogue inputs, by the last wave before the barrier (as tile_compute).
  constexpr int KU = C * MB;
  constexpr int kEpiWave = kWaves - 1;
  if (wave == kEpiWave) {
    f32x4 sx[KU], sg[C];
    const bool resid = io.resid;
#pragma unroll
    for (int u = 0; u < KU; ++u) {
      const int c = u / MB, rb = u % MB;
      const int col0 = kNB * (nb0 + c);
      const f32x4* src = zero4;
      if (resid) {
        src = (const f32x4*)(io.x_in + (size_t)(16 * rb + (lane >> 2)) * p.d + col0 + 4 * (lane & 3));
      } else if (step == STEP_QKV && col0 < 2 * p.d) {
        const int t = (col0 % p.d % p.Dh) / kNB;
        src = (const f32x4*)(p.rope + ((size_t)(16 * rb + (lane >> 2)) * (p.Dh / 2) + 8 * t + 2 * (lane & 3)) * 2);
      }
      sx[u] = ldg(opaque(src));
    }
#pragma unroll
    for (int c = 0; c < C; ++c)
      sg[c] = ldg(opaque(resid ? (const f32x4*)(io.g_next + kNB * (nb0 + c) + 8 * (lane & 1)) : zero4));
#pragma unroll
    for (int u = 0; u < KU; ++u) lds_st<f32x4>(lds + epi_off(C, MB, 4) + (size_t)u * 1024 + lane * 16, sx[u]);
#pragma unroll
    for (int c = 0; c < C; ++c) lds_st<f32x4>(lds + epi_off(C, MB, 4) + (size_t)(C * MB + c) * 1024 + lane * 16, sg[c]);
  }
  if (wave != 0) {
#pragma unroll
    for (int u = 0; u < D; ++u) load_w(u, u);
  }
  __builtin_amdgcn_sched_barrier(0);
  if (wait_phase >= 0) {
    const Sync sy = make_sync(p, lds_flag);
    trace_mark(sy, wait_phase, 0);
    if (!grid_wait(sy, wait_phase, p.G)) return false;
    trace_mark(sy, wait_phase, 1);
  }
  constexpr bool SSQR = MB <= 2;
  constexpr int SSQN = SSQR ? 8 : 1;
  f32x4 sr[SSQN];
  if constexpr (SSQR) {
    constexpr int QUADS = 4 * MB, CH = 256 / QUADS;
    const int q = threadIdx.x % QUADS, ch = threadIdx.x / QUADS;
    const int t0 = ch * p.d_nb / CH, t1 = (ch + 1) * p.d_nb / CH;
    const bool on = io.norm && p.ssq_regs;
#pragma unroll
    for (int k = 0; k < SSQN; ++k)
      sr[k] = ldg(opaque(on && t0 + k < t1 ? (const f32x4*)(io.ssq + (size_t)(t0 + k) * (16 * MB) + 4 * q) : zero4));
  }
#pragma unroll
  for (int u = 0; u < D; ++u) load_a(u, u);
  __builtin_amdgcn_s_waitcnt(0);
  lds_barrier();
  if (wave == 0) {
#pragma unroll
    for (int u = 0; u < D; ++u) load_w(u, u);
  }
  __builtin_amdgcn_sched_barrier(0);
  if (wait_phase >= 0 && p.trace != nullptr && threadIdx.x == 0)
    stg(p.trace + (size_t)blockIdx.x * pass_phases(p.L) * 8 + wait_phase * 8 + 3, (long long)wall_clock64());

  f32x4 acc[MB][C];
#pragma unroll
  for (int rb = 0; rb < MB; ++rb)
#pragma unroll
    for (int c = 0; c < C; ++c) acc[rb][c] = f32x4{0.f, 0.f, 0.f, 0.f};
  bf16x8 c136;
#pragma unroll
  for (int e = 0; e < 8; ++e) c136[e] = (bf16)136.0f;
  auto group = [&](int u) {  // the group in stage u, into acc
    f32x4 tmp[MB][C], corr[MB];
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) {
      corr[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < C; ++c) tmp[rb][c] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      bf16x8 b[C];
#pragma unroll
      for (int c = 0; c < C; ++c) b[c] = q4_operand(bw[u][c][t]);
#pragma unroll
      for (int rb = 0; rb < MB; ++rb) {
#pragma unroll
        for (int c = 0; c < C; ++c) tmp[rb][c] = mfma16x16x32(ba[u][t][rb], b[c], tmp[rb][c]);
        corr[rb] = mfma16x16x32(ba[u][t][rb], c136, corr[rb]);
      }
    }
#pragma unroll
    for (int c = 0; c < C; ++c) {
      const float sc = __uint_as_float((bs[u][c] & 0xFFFFu) << 16);  // the column's bf16 scale
#pragma unroll
      for (int rb = 0; rb < MB; ++rb) acc[rb][c] += sc * (tmp[rb][c] - corr[rb]);
    }
  };
  int i = 0;
  for (; i + D < ns; i += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      __builtin_amdgcn_sched_barrier(0);
      group(u);
      __builtin_amdgcn_sched_barrier(0);
      load_w(u, i + u + D);
      load_a(u, i + u + D);
    }
  }
  if (i < ns) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      __builtin_amdgcn_sched_barrier(0);
      group(u);
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (SSQR) {
    if (io.norm && p.ssq_regs) {
      constexpr int QUADS = 4 * MB;
      const int q = threadIdx.x % QUADS, ch = threadIdx.x / QUADS;
      f32x4 t = sr[0];
#pragma unroll
      for (int k = 1; k < SSQN; ++k) t += sr[k];
      *(f32x4*)&gl.part_ss[ch * 16 * MB + 4 * q] = t;
    }
  }
#pragma unroll
  for (int c = 0; c < C; ++c)
#pragma unroll
    for (int rb = 0; rb < MB; ++rb)
      lds_st<f32x4>(lds + tw_off() + ((size_t)((wave * C + c) * MB + rb) * 64 + lane) * 16, acc[rb][c]);
  __syncthreads();
  return true;
}

template <int MB, int C>
__device__ __forceinline__ bool tile_dispatch_q4(int cw, KParams& p, int step, int layer, int nb0, int wait_phase,
                                                 char* lds, GemmLds& gl, int* flag) {
  if constexpr (C >= 1) {
    if (cw == C) return tile_compute_q4<MB, C>(p, step, layer, nb0, wait_phase, lds, gl, flag);
    return tile_dispatch_q4<MB, C - 1>(cw, p, step, layer, nb0, wait_phase, lds, gl, flag);
  } else {
    return false;
  }
}

template <int MB, int C>
__device__ __forceinline__ bool tile_dispatch(int cw, KParams& p, int step, int layer, int nb0, int wait_phase,
                                              char* lds, GemmLds& gl, int* flag, int k0, int kn, int epi_in) {
  if constexpr (C >= 1) {
    if (cw == C) return tile_compute<MB, C>(p, step, layer, nb0, wait_phase, lds, gl, flag, k0, kn, epi_in);
    return tile_dispatch<MB, C - 1>(cw, p, step, layer, nb0, wait_phase, lds, gl, flag, k0, kn, epi_in);
  } else {
    return false;
  }
}

// Rotary embedding frequency of dim pair (j, j + Dh/2): theta^(-2j/Dh).
__device__ __forceinline__ float rope_inv_freq(int j, int Dh, float log2_theta) {
  return exp2f(-(2.0f * (float)j / (float)Dh) * log2_theta);
}

// RMSNorm scales of rows [0, Mp): 1 / sqrt(mean of squares + eps) from the
// per-16-column sums of squares the producing phase wrote, added in a fixed
// order; 0 for rows >= n.  When the tile held them in registers its chunk
// sums are in part_ss already.
// RMSNorm scales of rows [0, Mp) into gl.rstd from a version's sums of
// squares ssq [d/16][Mp] (added in a fixed order); 0 for rows >= n.
template <int MB>
__device__ __forceinline__ void row_rstd(KParams& p, const float* ssq, GemmLds& gl) {
  // thread t: rows 4 q .. 4 q + 3 (q = t % (ROWS / 4)) of the 16-column blocks
  // of chunk t / (ROWS / 4); 16-byte loads, a batch of them in flight at once
  // (a chunk's 4096 columns in one batch at 128 rows)
  constexpr int ROWS = 16 * MB, QUADS = ROWS / 4, CHK = kThreads / QUADS, BATCH = MB >= 8 ? 32 : 16;
  const int q = threadIdx.x % QUADS, ch = threadIdx.x / QUADS;
  const int dn = p.d_nb;
  const int t0 = ch * dn / CHK, t1 = (ch + 1) * dn / CHK;
  f32x4 ss = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int t = t0; t < t1; t += BATCH) {
    f32x4 v[BATCH];
#pragma unroll
    for (int k = 0; k < BATCH; ++k)
      v[k] = t + k < t1 ? ldg((const f32x4*)(ssq + (size_t)(t + k) * ROWS + 4 * q)) : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < BATCH; ++k) ss += v[k];
  }
  *(f32x4*)&gl.part_ss[ch * ROWS + 4 * q] = ss;
  __syncthreads();
  if (threadIdx.x < ROWS) {
    float t = 0.0f;
    for (int c = 0; c < CHK; ++c) t += gl.part_ss[c * ROWS + threadIdx.x];
    gl.rstd[threadIdx.x] = threadIdx.x < p.n ? 1.0f / sqrtf(t * p.inv_d + p.eps) : 0.0f;
  }
  __syncthreads();
}

template <int MB>
__device__ __forceinline__ void row_scales(KParams& p, const StepIo& io, GemmLds& gl) {
  constexpr int ROWS = 16 * MB;
  if (MB <= 2 && p.ssq_regs) {
    constexpr int CH = 256 / (4 * MB);
    if (threadIdx.x < ROWS) {
      float t = 0.0f;
      for (int c = 0; c < CH; ++c) t += gl.part_ss[c * ROWS + threadIdx.x];
      gl.rstd[threadIdx.x] = threadIdx.x < p.n ? 1.0f / sqrtf(t * p.inv_d + p.eps) : 0.0f;
    }
    __syncthreads();
    return;
  }
  row_rstd<MB>(p, io.ssq, gl);
}

// Epilogue of one accumulator tile ("unit": block c of the tile x row block
// rb, 16 x 16).  The unit's sum is the nsum partial tiles in LDS added in
// order (the four waves' partials, or a split-K group's partial sums in
// slice order); lane l holds rows 16 rb + 4 (l / 16) + i, i < 4, column
// l % 16.
// Outputs are written with device-coherent stores.
template <int MB, int EPI>
__device__ __forceinline__ void epilogue_unit(KParams& p, const StepIo& io, const char* lds, int cw, int c, int rb,
                                              int nb, GemmLds& gl, int nsum) {
  const int lane = threadIdx.x & 63, j = lane & 15, q4 = lane >> 4;
  const int unit = c * MB + rb;
  f32x4 s = lds_ld<f32x4>(lds + tw_off() + ((size_t)unit * 64 + lane) * 16);
#pragma unroll
  for (int w = 1; w < kWaves; ++w)
    if (w < nsum) s += lds_ld<f32x4>(lds + tw_off() + ((size_t)(w * cw * MB + unit) * 64 + lane) * 16);
  float v[4] = {s[0], s[1], s[2], s[3]};
  const int rr0 = 4 * q4;  // first row of this lane inside the row block
  if constexpr (EPI == EPI_QKV || EPI == EPI_SWIGLU) {  // the norm's per-row scale
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] *= gl.rstd[16 * rb + rr0 + i];
  }
  const char* epi = lds + epi_off(cw, MB, nsum);
  const int col = kNB * nb + j;
  if constexpr (EPI == EPI_QKV) {
    const int d = p.d, dh = p.Dh;
    if (kNB * nb < 2 * d) {
      // q or k: this block holds dims [8t, 8t+8) (lanes j < 8) and their
      // rotary partners + Dh/2 (lanes j >= 8) of one head.
      const int part = (kNB * nb) / d, cq = (kNB * nb) % d, hh = cq / dh, t = (cq % dh) / kNB;
      const int dim = 8 * t + (j & 7) + (j < 8 ? 0 : dh / 2);
      bf16* base = part == 0 ? io.q + hh * dh : io.kc + (size_t)hh * p.cap * dh;
      const char* csu = epi + (size_t)unit * 1024;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int rr = rr0 + i, r = 16 * rb + rr;
        const float2 cs = lds_ld<float2>(csu + (size_t)(rr * 8 + (j & 7)) * 8);
        const float partner = dpp_f<kDppRowRor8>(v[i]);
        const float outv = j < 8 ? v[i] * cs.x - partner * cs.y : v[i] * cs.x + partner * cs.y;
        const float nxt = dpp_f<kDppRowShl1>(outv);
        if (r < p.n && (j & 1) == 0) {
          bf16* dst = part == 0 ? base + (size_t)r * d : base + (size_t)(p.prefix_len + p.m0 + r) * dh;
          st_coherent_bf2(dst + dim, outv, nxt);
        }
      }
    } else {
      // v: the cache holds V transposed per head ([Dh][cap]); this lane's
      // four rows are four consecutive slots of one dim
      const int cv = col - 2 * d, hh = cv / dh, dim = cv % dh;
      bf16* vrow = io.vc + ((size_t)hh * dh + dim) * p.cap + p.prefix_len + p.m0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 16 * rb + rr0 + i;
        if (r < p.n) st_coherent_bf(vrow + r, v[i]);
      }
    }
  } else if constexpr (EPI == EPI_RESID) {
    const char* xu = epi + (size_t)unit * 1024;
    const float g = bf2f(lds_ld<bf16>(epi + (size_t)(cw * MB + c) * 1024 + 16 * (j >> 3) + 2 * (j & 7)));
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rr = rr0 + i, r = 16 * rb + rr;
      const float xn = r < p.n ? lds_ld<float>(xu + (size_t)(rr * 16 + j) * 4) + v[i] : 0.0f;
      const float xn1 = dpp_f<kDppRowShl1>(xn);
      if (r < p.n && (j & 1) == 0) st_coherent2(io.x_out + (size_t)r * p.d + col, xn, xn1);
      const float xg = xn * g;
      const float xg1 = dpp_f<kDppRowShl1>(xg);
      if (r < p.n && (j & 1) == 0) st_coherent_bf2(io.xg_out + frag_off(r, col, MB), xg, xg1);
      const float sq = row16_sum(xn * xn);  // sum of squares over the block's 16 columns
      if (j == 0 && r < p.n) st_coherent(io.ssq_out + (size_t)nb * p.Mp + r, sq);
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    const int f = 8 * nb + (j & 7);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 16 * rb + rr0 + i;
      const float up = dpp_f<kDppRowRor8>(v[i]);
      const float hv = v[i] / (1.0f + expf(-v[i])) * up;
      const float nxt = dpp_f<kDppRowShl1>(hv);
      if (r < p.n && j < 8 && (j & 1) == 0) st_coherent_bf2(io.h + frag_off(r, f, MB), hv, nxt);
    }
  } else {  // EPI_LOGITS
    const bool vcol = col < p.V;
    // (with candidate summaries the end of the pass reads the stored rows
    // back: device-coherent stores)
    const bool summ = p.cand != nullptr;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 16 * rb + rr0 + i;
      const bool valid = vcol && r < p.n;
      if (valid && p.logits != nullptr && r >= p.row_lo) {
        float* dst = p.logits + (size_t)(r - p.row_lo) * p.V + col;
        if (summ)
          st_coherent(dst, v[i]);
        else
          stg(dst, v[i]);
      }
      float mv = valid ? v[i] : -INFINITY;
      int mi = valid ? col : 0x7fffffff;
      row16_argmax(mv, mi);  // argmax over the block's 16 columns
      // the block's sum of exp(logit - its max), for the softmax normaliser
      const float se = summ ? row16_sum(valid ? expf(v[i] - mv) : 0.0f) : 0.0f;
      if (j == 0) {
        gl.red_v[r][c] = mv;
        gl.red_i[r][c] = mi;
        gl.red_s[r][c] = se;
      }
    }
  }
}

// After all argmax partials are in: greedy token per node and the accept walk
// (§3.2): node i is reachable when its parent is and its draft token equals
// the target's token after the parent; the result is the deepest reachable
// node (lowest index among equally deep ones).
//
// One workgroup, so every dependent step is paid once per pass: the tree and
// all of a wave's argmax partials are loaded in one round trip, the rows'
// reductions are interleaved, and reachability is found by pointer jumping
// (ceil(log2 n) rounds over all nodes at once) instead of a serial walk.
// (LDS hand-offs only: lds_barrier, which leaves the global stores in flight.)
__device__ __forceinline__ void finish_walk(KParams& p, int entries, GemmLds& gl) {
  const int wave = wave_index(), lane = threadIdx.x & 63;
  const int n = p.n;
  // the tree (written by the first phase): one node per thread (n <= 128)
  const int me = threadIdx.x;
  const bool mine = me < n;
  const int t_tok = ldg(p.tree + (mine ? me : 0));
  const int t_par = ldg(p.tree + 128 + (mine ? me : 0));
  const int t_dep = ldg(p.tree + 256 + (mine ? me : 0));
  constexpr int RB = 8;  // rows per wave whose partials are loaded together
  for (int r0 = wave; r0 < n; r0 += kWaves * RB) {
    float mv[RB];
    int mi[RB];
#pragma unroll
    for (int k = 0; k < RB; ++k) {
      mv[k] = -INFINITY;
      mi[k] = 0x7fffffff;
    }
    for (int t0 = 0; t0 < entries; t0 += 4 * 64) {
      float v[RB][4];
      int ix[RB][4];
#pragma unroll
      for (int k = 0; k < RB; ++k)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int t = t0 + 64 * u + lane, r = r0 + kWaves * k;
          const bool on = t < entries && r < n;
          v[k][u] = on ? ld_coherent(&p.lm_val[(size_t)r * p.G + t]) : -INFINITY;
          ix[k][u] = on ? ld_coherent(&p.lm_idx[(size_t)r * p.G + t]) : 0x7fffffff;
        }
#pragma unroll
      for (int k = 0; k < RB; ++k)
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (v[k][u] > mv[k] || (v[k][u] == mv[k] && ix[k][u] < mi[k])) {
            mv[k] = v[k][u];
            mi[k] = ix[k][u];
          }
    }
    // across the wave: rows of 16 lanes on DPP, then lanes 16 and 32 apart
#pragma unroll
    for (int k = 0; k < RB; ++k) row16_argmax(mv[k], mi[k]);
#pragma unroll
    for (int off = 16; off <= 32; off *= 2) {
#pragma unroll
      for (int k = 0; k < RB; ++k) {
        const float ov = __shfl_xor(mv[k], off, kWave);
        const int oi = __shfl_xor(mi[k], off, kWave);
        if (ov > mv[k] || (ov == mv[k] && oi < mi[k])) {
          mv[k] = ov;
          mi[k] = oi;
        }
      }
    }
#pragma unroll
    for (int k = 0; k < RB; ++k) {
      const int r = r0 + kWaves * k;
      if (lane == 0 && r < n) {
        stg(p.amax + r, mi[k]);
        gl.amax[r] = mi[k];
      }
    }
  }
  if (mine) {
    gl.tok[me] = t_tok;
    gl.par[me] = t_par;
    gl.dep[me] = t_dep;
  }
  lds_barrier();
  // reach[i]: AND of ok over node i and its ancestors below jump[i], where
  // ok(i) = (token of i == greedy token after its parent), ok(root) = 1;
  // each round doubles the span (jump[i] <- jump[jump[i]]) until every
  // jump[] is the root, whose reach is 1.
  if (mine) {
    gl.reach[me] = me == 0 ? 1 : (t_tok == gl.amax[t_par > 0 ? t_par : 0] ? 1 : 0);
    gl.jump[me] = me == 0 ? 0 : t_par;
  }
  lds_barrier();
  for (int span = 1; span < n; span *= 2) {
    int rv = 0, jv = 0;
    if (mine) {
      const int j = gl.jump[me];
      rv = gl.reach[me] & gl.reach[j];
      jv = gl.jump[j];
    }
    lds_barrier();
    if (mine) {
      gl.reach[me] = rv;
      gl.jump[me] = jv;
    }
    lds_barrier();
  }
  // deepest reachable node, lowest index first: max of (depth, 127 - i)
  if (wave == 0) {
    int key = -1;
    for (int i = lane; i < n; i += 64)
      if (gl.reach[i]) key = max(key, (gl.dep[i] << 8) | (127 - i));
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) key = max(key, __shfl_xor(key, off, kWave));
    if (lane == 0) {
      const int best = 127 - (key & 255), best_depth = key >> 8;
      for (int i = best; i >= 0; i = gl.par[i]) gl.jump[gl.dep[i]] = i;  // the path, by depth
      gl.walk_len = best_depth;
      stg(p.accept_len, best_depth);
      stg(p.next_token, gl.amax[best]);
    }
  }
  lds_barrier();
  {
    const int best_depth = gl.walk_len;
    for (int k = threadIdx.x; k < n; k += kThreads) stg(p.path + k, k <= best_depth ? gl.jump[k] : -1);
  }
  lds_barrier();
}

// (max, normaliser, argmax) of a set of logits merged with another set's:
// the normalisers are sums of exp(logit - own max), rescaled to the larger
// maximum; the argmax keeps the lowest index among equal maxima.
__device__ __forceinline__ void softmax_merge(float& m, float& s, int& ix, float om, float os, int oi) {
  const float mn = fmaxf(m, om);
  s = (m == -INFINITY ? 0.0f : s * expf(m - mn)) + (om == -INFINITY ? 0.0f : os * expf(om - mn));
  if (om > m || (om == m && oi < ix)) ix = oi;
  m = mn;
}

// Candidate summaries of the computed rows (llmcad_extend_tree_candidates),
// by the workgroup that completes the LM head's argmax, at the end of the
// pass: per row, the workgroups' (max, argmax, normaliser) partials are
// merged (one wave, in a fixed order), the stored logits row is scanned once
// for every token whose probability exp(logit - max) / normaliser exceeds
// the threshold, and the argmax and those tokens are written sorted by
// probability, higher first (ties: lower token first).  `lds`: the GEMM
// tiles' region, free once the phase's tiles are done.
__device__ __attribute__((noinline, not_tail_called)) void finish_candidates(KParams& pin, int entries, char* lds) {
  KParams& p = uniform_params(pin);
  const int wave = wave_index(), lane = threadIdx.x & 63;
  float* sm = (float*)lds;       // the row's max and normaliser
  int* si = (int*)(lds + 64);    // its argmax and the candidate count
  int* ctok = (int*)(lds + 1024);
  float* cprob = (float*)(lds + 1024 + 4 * LLMCAD_CAND_MAX);
  const int G = p.G, V = p.V;
  for (int r = p.row_lo; r < p.n; ++r) {
    if (wave == 0) {
      float m = -INFINITY, s = 0.0f;
      int ix = 0x7fffffff;
      for (int t = lane; t < entries; t += 64)
        softmax_merge(m, s, ix, ld_coherent(&p.lm_val[(size_t)r * G + t]), ld_coherent(&p.lm_sum[(size_t)r * G + t]),
                      ld_coherent(&p.lm_idx[(size_t)r * G + t]));
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) {
        const float om = __shfl_xor(m, off, kWave), os = __shfl_xor(s, off, kWave);
        const int oi = __shfl_xor(ix, off, kWave);
        softmax_merge(m, s, ix, om, os, oi);
      }
      if (lane == 0) {
        sm[0] = m;
        sm[1] = s;
        si[0] = ix;
        si[1] = 0;
      }
    }
    __syncthreads();
    const float M = sm[0], S = sm[1], thr = p.cand_thr;
    const int amax = si[0];
    const float* row = p.logits + (size_t)(r - p.row_lo) * V;
    for (int v = threadIdx.x; v < V; v += kThreads) {
      const float pr = expf(ld_coherent(row + v) - M) / S;
      if (pr > thr || v == amax) {
        const int k = atomicAdd(&si[1], 1);
        if (k < LLMCAD_CAND_MAX) {
          ctok[k] = v;
          cprob[k] = pr;
        }
      }
    }
    __syncthreads();
    const int cnt = si[1];
    llmcad_candidates* rec = p.cand + (r - p.row_lo);
    if (wave == 0) {
      if (cnt <= LLMCAD_CAND_MAX && lane < cnt) {
        const float mine = cprob[lane];
        const int mt = ctok[lane];
        int rank = 0;
        for (int j = 0; j < cnt; ++j) rank += (cprob[j] > mine || (cprob[j] == mine && ctok[j] < mt)) ? 1 : 0;
        stg(&rec->tok[rank], mt);
        stg(&rec->prob[rank], mine);
      }
      if (lane == 0) {
        stg(&rec->count, cnt <= LLMCAD_CAND_MAX ? cnt : -1);
        stg(&rec->argmax, amax);
        stg(&rec->max_logit, M);
        stg(&rec->sum_exp, S);
      }
    }
    __syncthreads();
  }
}

// The epilogue of one tile (blocks [nb0, nb0 + cw)): the waves take its
// units in turn.  The LM head also folds the tile's per-block argmax into
// the workgroup's running argmax per row.  A function of its own so that its
// registers are allocated apart from the streaming loop's.
template <int MB, int EPI>
__device__ __attribute__((noinline, not_tail_called)) void finish_tile(KParams& pin, int step, int layer, int nb0,
                                                                      int cw, char* lds, GemmLds& gl, int nsum) {
  KParams& p = uniform_params(pin);
  step = wave_uniform(step);
  layer = wave_uniform(layer);
  nb0 = wave_uniform(nb0);
  cw = wave_uniform(cw);
  nsum = wave_uniform(nsum);
  const StepIo io = step_io<EPI>(p, step, layer);
  if constexpr (EPI == EPI_QKV || EPI == EPI_SWIGLU) row_scales<MB>(p, io, gl);
  const int units = cw * MB;
  for (int u = wave_index(); u < units; u += kWaves) {
    const int c = u / MB, rb = u % MB;
    epilogue_unit<MB, EPI>(p, io, lds, cw, c, rb, nb0 + c, gl, nsum);
  }
  if constexpr (EPI == EPI_LOGITS) {
    __syncthreads();
    const bool summ = p.cand != nullptr;
    for (int r = threadIdx.x; r < 16 * MB; r += kThreads) {
      float mv = gl.best_v[r];
      int mi = gl.best_i[r];
      float ms = gl.best_s[r];
      for (int c = 0; c < cw; ++c) {
        const float v = gl.red_v[r][c];
        const int i = gl.red_i[r][c];
        if (summ) {  // the normalisers, relative to the larger of the two maxima
          const float mn = fmaxf(mv, v);
          ms = (mv == -INFINITY ? 0.0f : ms * expf(mv - mn)) + (v == -INFINITY ? 0.0f : gl.red_s[r][c] * expf(v - mn));
        }
        if (v > mv || (v == mv && i < mi)) {
          mv = v;
          mi = i;
        }
      }
      gl.best_v[r] = mv;
      gl.best_i[r] = mi;
      gl.best_s[r] = ms;
    }
  }
  __syncthreads();
}

// ---- split-K (projections with one column block per workgroup at 64 or
// more rows: every workgroup would read the whole activation matrix per
// block of weights)
//
// Groups of S consecutive workgroups (virtual index) share a group of column
// blocks; workgroup s of a group computes every block of the group over the
// k-steps [s ks/S, (s+1) ks/S), so it reads 1/S of the activations for the
// same weight bytes.  Each stores its partial tiles (its waves' partials
// added in wave order), counts its arrival on the group's counter, and then
// finishes 1/S of the group's blocks: it waits for the group, adds the S
// partial tiles of each of its units in slice order (bit-reproducible) and
// runs the step's epilogue.

// The tile's partial sums (its partial tiles in LDS, added in slot order)
// to dst: unit u = c MB + rb of the tile at dst + u KiB, lane l's 16 bytes
// at + 16 l.  Device-coherent stores: the region is reused by every split
// phase of the pass.
template <int MB>
__device__ __forceinline__ void split_store(const char* lds, int cw, float* dst) {
  const int lane = threadIdx.x & 63;
  const int nsl = tile_slots(cw, MB);
  for (int u = wave_index(); u < cw * MB; u += kWaves) {
    f32x4 s = lds_ld<f32x4>(lds + tw_off() + ((size_t)u * 64 + lane) * 16);
#pragma unroll
    for (int w = 1; w < kWaves; ++w)
      if (w < nsl) s += lds_ld<f32x4>(lds + tw_off() + ((size_t)(w * cw * MB + u) * 64 + lane) * 16);
    float* q = dst + ((size_t)u * 64 + lane) * 4;
    st_coherent2(q, s[0], s[1]);
    st_coherent2(q + 2, s[2], s[3]);
  }
}

// Waits (wave 0 polls) until the counter reaches `want`; false (to all
// threads) if the bounded spin ran out (the pass status is then set).
__device__ __forceinline__ bool counter_wait(const Sync& s, const int* cnt, int want) {
  if (threadIdx.x < 64) {
    int ok = 1;
    if (s.limit < 0) {
      ok = 0;
    } else {
      int spins = 0;
      while (ld_coherent(cnt) < want) {
        __builtin_amdgcn_s_sleep(1);
        if (++spins > s.limit) {
          ok = 0;
          break;
        }
      }
    }
    if (!ok && threadIdx.x == 0) st_coherent(s.status, 1);
    if (threadIdx.x == 0) *s.lds_flag = ok;
  }
  lds_barrier();
  const bool ok = *s.lds_flag != 0;
  lds_barrier();
  return ok;
}

// One split-K phase of a residual step (O or down).  Each group counts its
// arrivals on a counter of its own step, S per layer (the step's S is fixed
// for the pass), so the counter reaches S (layer + 1) exactly when the group
// has arrived in this layer.
template <int MB, int EPI>
__device__ __attribute__((noinline, not_tail_called)) bool split_phase(KParams& pin, int step, int layer,
                                                                      int phase, char* lds, GemmLds& gl,
                                                                      int* lds_flag) {
  KParams& p = uniform_params(pin);
  step = wave_uniform(step);
  layer = wave_uniform(layer);
  phase = wave_uniform(phase);
  const Sync sy = make_sync(p, lds_flag);
  const StepPlan& sp = p.step[step];
  constexpr int CM = MB <= 2 ? 8 : MB == 4 ? LLMCAD_TILE_BLOCKS_MB4 : LLMCAD_TILE_BLOCKS_MB8;
  const int S = wave_uniform(sp.split), G = p.G, NG = G / S;
  const int nbk = sp.nblocks, ks = sp.ksteps;
  const int vw = virtual_wg(G);
  const int g = vw / S, sl = vw % S;
  const int glo = wave_uniform((int)((long)g * nbk / NG));
  const int ghi = wave_uniform((int)((long)(g + 1) * nbk / NG));
  const int bstride = (nbk + NG - 1) / NG;  // partial-tile slots per workgroup, in blocks
  const int k0 = sl * ks / S, k1 = (sl + 1) * ks / S;
  const int wave = wave_index(), lane = threadIdx.x & 63;
  constexpr int U = MB * 256;  // floats of one block's partial tiles
  int* cnt = p.grp_cnt + (step == STEP_DOWN ? kPassMaxGrid / 2 : 0) + g;
  if (glo >= ghi) {  // (no blocks: the host splits only steps with a block per group)
    trace_mark(sy, phase, 0);
    if (!grid_wait(sy, phase, G)) return false;
    trace_mark(sy, phase, 1);
    return true;
  }
  float* mine = p.part + (size_t)vw * bstride * U;
  for (int b0 = glo; b0 < ghi; b0 += CM) {
    const int cw = ghi - b0 < CM ? ghi - b0 : CM;
    const bool first = b0 == glo;
    if (!tile_dispatch<MB, CM>(cw, p, step, layer, b0, first ? phase : -1, lds, gl, lds_flag, k0, k1 - k0, 0))
      return false;
    if (first) trace_mark(sy, phase, 4);
    split_store<MB>(lds, cw, mine + (size_t)(b0 - glo) * U);
    __syncthreads();  // (the next tile and the finish reuse the LDS)
  }
  // This workgroup's partial tiles have completed; count its arrival.
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) atomic_add_dev(cnt, 1);
  const int B = ghi - glo;
  const int olo = glo + sl * B / S, ohi = glo + (sl + 1) * B / S;  // the blocks it finishes
  if (olo >= ohi) {
    trace_mark(sy, phase, 5);
    return true;
  }
  const TileIn io = tile_in(p, step, layer);
  for (int c0 = olo; c0 < ohi; c0 += CM) {
    const int cw = wave_uniform(ohi - c0 < CM ? ohi - c0 : CM);
    char* epi = lds + epi_off(cw, MB, S);
    // epilogue inputs (written two or more phases ago): the residual rows of
    // each unit and the next norm's gains, straight to LDS, before the wait
    if (wave == kWaves - 1) {
      for (int u = 0; u < cw * MB; ++u) {
        const int c = u / MB, rb = u % MB;
        dma16(io.x_in + (size_t)(16 * rb + (lane >> 2)) * p.d + kNB * (c0 + c) + 4 * (lane & 3),
              epi + (size_t)u * 1024);
      }
      for (int c = 0; c < cw; ++c) dma16(io.g_next + kNB * (c0 + c) + 8 * (lane & 1), epi + (size_t)(cw * MB + c) * 1024);
    }
    if (c0 == olo && !counter_wait(sy, cnt, S * (layer + 1))) return false;
    // the group's S partial tiles of each unit -> LDS slots [t][c][rb]
    for (int it = wave; it < S * cw * MB; it += kWaves) {
      const int t = it / (cw * MB), u = it % (cw * MB);
      const float* src = p.part + ((size_t)(g * S + t) * bstride + (c0 - glo)) * U + ((size_t)u * 64 + lane) * 4;
      const float2 a = ld_coherent2(src), b = ld_coherent2(src + 2);
      lds_st<f32x4>(lds + tw_off() + ((size_t)(t * cw * MB + u) * 64 + lane) * 16, f32x4{a.x, a.y, b.x, b.y});
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    finish_tile<MB, EPI>(p, step, layer, c0, cw, lds, gl, S);
  }
  trace_mark(sy, phase, 5);
  return true;
}

// One GEMM phase: this workgroup's run of blocks, in tiles over the full K
// (K-split tiles of up to 8, 6 or 4 blocks at 32, 64 or 128 rows; row-split
// tiles of up to 8 where a run exceeds one K-split tile at 64+ rows; 4-bit
// tiles of up to 6, 2 or 1), each followed by its epilogue.  The LM head then
// publishes the workgroup's argmax per row, and the last workgroup to do so
// runs the accept walk.
template <int MB, int EPI, int CM2 = 8>
__device__ __attribute__((noinline, not_tail_called)) bool gemm_phase(KParams& pin, int step, int layer,
                                                                     int phase, char* lds, GemmLds& gl,
                                                                     int* lds_flag) {
  KParams& p = uniform_params(pin);
  step = wave_uniform(step);
  layer = wave_uniform(layer);
  phase = wave_uniform(phase);
  const Sync sy = make_sync(p, lds_flag);
  const StepPlan& sp = p.step[step];
  // (CM2: 8, or 9 for a step marked wide; the LM head keeps 8, its per-block
  // argmax slots)
  constexpr int CM = MB <= 2 ? CM2 : MB == 4 ? LLMCAD_TILE_BLOCKS_MB4 : LLMCAD_TILE_BLOCKS_MB8;
  static_assert(wl_off(CM, MB, tile_slots(CM, MB)) <= kGemmLdsBytes,
                "a tile's partial sums and epilogue inputs fit the LDS");
  static_assert(EPI != EPI_LOGITS || CM2 <= 8, "the LM head's per-block argmax slots");
  // 4-bit tiles hold a second set of accumulators (each group's partial sums)
  constexpr int CMQ = MB <= 2 ? 6 : MB == 4 ? 2 : 1;
  // Row-split tiles (up to 8 blocks) for a workgroup of a pass of 64+ rows
  // whose blocks do not fit one K-split tile: it then reads the activations
  // once instead of once per tile (where one K-split tile holds them all,
  // that tile is faster: no barrier per k-step).
  constexpr int CMR = 8;
  static_assert(MB < 4 || wl_off(CMR, MB, 1) <= kGemmLdsBytes, "a row-split tile fits the LDS");
  const bool q4 = wave_uniform(sp.q4) != 0;
  const int nbk = sp.nblocks, G = p.G;
  const int vw = virtual_wg(G);
  const int lo = wave_uniform((int)((long)vw * nbk / G));
  const int hi = wave_uniform((int)((long)(vw + 1) * nbk / G));
  const bool rows = MB >= 4 && !q4 && wave_uniform(p.row_tiles) != 0 && hi - lo > CM;
  const int cm = q4 ? CMQ : rows ? CMR : CM;
  if constexpr (EPI == EPI_LOGITS) {
    for (int r = threadIdx.x; r < 16 * MB; r += kThreads) {
      gl.best_v[r] = -INFINITY;
      gl.best_i[r] = 0x7fffffff;
      gl.best_s[r] = 0.0f;
    }
  }
  if (lo >= hi) {
    // The barrier counts arrivals: it is exact only if every workgroup waits
    // at every phase before it arrives again, work or no work.
    trace_mark(sy, phase, 0);
    if (!grid_wait(sy, phase, G)) return false;
    trace_mark(sy, phase, 1);
  }
  for (int b0 = lo; b0 < hi; b0 += cm) {
    const int cw = hi - b0 < cm ? hi - b0 : cm;
    const bool first = b0 == lo;
    bool ok;
    if constexpr (MB >= 4) {
      ok = q4     ? tile_dispatch_q4<MB, CMQ>(cw, p, step, layer, b0, first ? phase : -1, lds, gl, lds_flag)
           : rows ? tile_dispatch_rows<MB, CMR>(cw, p, step, layer, b0, first ? phase : -1, lds, lds_flag)
                  : tile_dispatch<MB, CM>(cw, p, step, layer, b0, first ? phase : -1, lds, gl, lds_flag, 0,
                                          sp.ksteps, 1);
    } else {
      ok = q4 ? tile_dispatch_q4<MB, CMQ>(cw, p, step, layer, b0, first ? phase : -1, lds, gl, lds_flag)
              : tile_dispatch<MB, CM>(cw, p, step, layer, b0, first ? phase : -1, lds, gl, lds_flag, 0,
                                      sp.ksteps, 1);
    }
    if (!ok) return false;
    if (first) trace_mark(sy, phase, 4);
    finish_tile<MB, EPI>(p, step, layer, b0, cw, lds, gl, q4 ? 4 : rows ? 1 : tile_slots(cw, MB));
  }
  trace_mark(sy, phase, 5);
  if constexpr (EPI == EPI_LOGITS) {
    __syncthreads();
    for (int r = threadIdx.x; r < 16 * MB; r += kThreads) {
      st_coherent(&p.lm_val[(size_t)r * G + blockIdx.x], gl.best_v[r]);
      st_coherent(&p.lm_idx[(size_t)r * G + blockIdx.x], gl.best_i[r]);
      if (p.cand != nullptr) st_coherent(&p.lm_sum[(size_t)r * G + blockIdx.x], gl.best_s[r]);
    }
    if (arrive_last(p.lm_cnt, G, lds_flag)) {
      if (p.m0 == 0) {
        trace_mark(sy, phase, 6);
        finish_walk(p, G, gl);
        trace_mark(sy, phase, 7);
      }
      if (p.cand != nullptr) finish_candidates(p, G, lds);
    }
  }
  return true;
}

// ------------------------------------------------------------------ attention

// The cache holds K row-major per head ([cap][DH]) and V transposed per head
// ([DH][cap]), so that both operands of the attention's matrix products load
// straight from memory in MFMA fragment order, 16 bytes per lane, with no
// staging or transposition in between:
//  - K is the A operand of S^T = K q^T (16 keys x 32 dims per MFMA).  Key
//    block b of a 32-key step at key0 puts key key0 + 8 (r / 4) + 4 b + r % 4
//    in its row r, so that lane (li, g) of the result holds the scores of keys
//    key0 + 8 g + 4 b + i (i < 4) for query row li;
//  - V^T is the A operand of O^T = V^T P^T (16 dims x 32 keys): lane (li, g)
//    holds dim 16 db + li for keys key0 + 8 g .. + 7 -- exactly the keys whose
//    scores it holds, so the probabilities go from the S result into the PV
//    product's B operand without leaving the lane.
template <int DH>
struct AttnStep {
  static constexpr int NS = DH / 32;         // 32-dim k-steps of S^T
  static constexpr int NB = DH / 16;         // 16-dim blocks of O^T
  static constexpr int LOADS = 2 * NS + NB;  // 16-byte loads per lane (1 KiB per wave each)
  bf16x8 f[LOADS];                           // K block b, k-step s at b NS + s; V^T block db at 2 NS + db
};

// Steps of a unit fetched before the phase's barrier.  Wave 0 polls the
// barrier and issues no load before it has seen it (a poll waits for every
// older load of its wave), so its first W0 steps are copied straight to LDS
// by wave 1; wave 1 holds its first two steps in registers; waves 2 and 3
// hold two in registers and the next W23 in LDS.  The LDS slots (one step
// each) are laid out wave 0's, then wave 2's, then wave 3's.
template <int DH>
struct AttnPrefetch {
  static constexpr int REG = 2;
  static constexpr int STEP_BYTES = AttnStep<DH>::LOADS * 1024;  // one wave's step
  static constexpr int SLOTS0 = kGemmLdsBytes / STEP_BYTES;
  static constexpr int SLOTS = SLOTS0 < 16 ? SLOTS0 : 16;
  static constexpr int W0 = SLOTS / 2 < 6 ? SLOTS / 2 : 6;
  static constexpr int W23 = (SLOTS - W0) / 2;
  static constexpr int STEPS = W0 + REG + 2 * (REG + W23);  // per unit
  // steps in registers and in LDS of wave w, and the first LDS slot of its share
  __device__ static int reg(int w) { return w == 0 ? 0 : REG; }
  __device__ static int lds(int w) { return w == 0 ? W0 : w == 1 ? 0 : W23; }
  __device__ static int slot0(int w) { return w == 0 ? 0 : w == 2 ? W0 : W0 + W23; }
};

// Source of load e of the 32-key step at key0 for this lane (the zero line
// for keys at or past lim).  kc: the head's K [cap][DH]; vt: its V^T [DH][cap]
// (cap a multiple of 8, so a lane's 8 keys never cross a row of V^T).
template <int DH>
__device__ __forceinline__ const bf16x8* attn_src(const bf16* kc, const bf16* vt, int cap, int key0, int lim,
                                                  const bf16x8* zero, int e) {
  const int lane = threadIdx.x & 63, li = lane & 15, g = lane >> 4;
  constexpr int NS = AttnStep<DH>::NS;
  if (e < 2 * NS) {
    const int b = e / NS, s = e % NS;
    const int key = key0 + 8 * (li >> 2) + 4 * b + (li & 3);
    return opaque(key < lim ? (const bf16x8*)(kc + (size_t)key * DH + 32 * s + 8 * g) : zero);
  }
  const int kv = key0 + 8 * g;
  return opaque(kv < lim ? (const bf16x8*)(vt + (size_t)(16 * (e - 2 * NS) + li) * cap + kv) : zero);
}

template <int DH>
__device__ __forceinline__ void attn_load(AttnStep<DH>& R, const bf16* kc, const bf16* vt, int cap, int key0, int lim,
                                          const bf16x8* zero) {
#pragma unroll
  for (int e = 0; e < AttnStep<DH>::LOADS; ++e) R.f[e] = ldg(attn_src<DH>(kc, vt, cap, key0, lim, zero, e));
}

// The step's loads copied straight to LDS: load e lands at buf + e KiB (lane
// l's 16 bytes at + 16 l).
template <int DH>
__device__ __forceinline__ void attn_copy(char* buf, const bf16* kc, const bf16* vt, int cap, int key0, int lim,
                                          const bf16x8* zero) {
#pragma unroll
  for (int e = 0; e < AttnStep<DH>::LOADS; ++e) dma16(attn_src<DH>(kc, vt, cap, key0, lim, zero, e), buf + e * 1024);
}

template <int DH>
__device__ __forceinline__ void attn_from_lds(AttnStep<DH>& R, const char* buf) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int e = 0; e < AttnStep<DH>::LOADS; ++e) R.f[e] = lds_ld<bf16x8>(buf + e * 1024 + lane * 16);
}

// One 32-key step for the 16 query rows of a unit: S^T on the matrix cores,
// the mask (the prefix, then the tree's slots of the row's ancestors-or-self;
// keys at or past lim are not visible), the online softmax in the log2 domain,
// and O^T += V^T P^T with P split into two bf16 halves (hi + lo, ~16
// significant bits).  V entries of keys at or past lim inside a loaded piece
// are zeroed: the cache there may hold anything, and 0 x NaN is NaN.
template <int DH>
__device__ __forceinline__ void attn_compute(const AttnStep<DH>& R, const bf16x8 (&qf)[DH / 32],
                                             const uint32_t (&anc)[4], int key0, int P, int lim, float scale_log2,
                                             float& m_run, float& l_run, f32x4 (&oacc)[DH / 16]) {
  constexpr int NS = AttnStep<DH>::NS, NB = AttnStep<DH>::NB;
  const int lane = threadIdx.x & 63, g = lane >> 4;
  f32x4 sc[2];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    sc[b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NS; ++s) sc[b] = mfma16x16x32(R.f[b * NS + s], qf[s], sc[b]);
  }
  // With one wave per SIMD a step costs what its instructions cost to issue:
  // a step of prefix keys only (most of them) skips the mask, and the others
  // take it branch-free (bitwise, not short-circuit).
  float sv[8];
  float mx = -INFINITY;
  if (key0 + 32 <= P && key0 + 32 <= lim) {  // (wave-uniform)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      sv[e] = sc[e >> 2][e & 3] * scale_log2;
      mx = fmaxf(mx, sv[e]);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int pos = key0 + 8 * g + e;
      const int t = pos - P < 0 ? 0 : pos - P;  // (tree slot; any in-range index for prefix keys)
      const uint32_t w = anc[(t >> 5) & 3];
      const uint32_t vis = (uint32_t)(pos < lim) & ((uint32_t)(pos < P) | ((w >> (t & 31)) & 1u));
      sv[e] = vis != 0u ? sc[e >> 2][e & 3] * scale_log2 : -INFINITY;
      mx = fmaxf(mx, sv[e]);
    }
  }
  mx = col4_max(mx);
  const float m_new = fmaxf(m_run, mx);
  const float m_use = m_new == -INFINITY ? 0.0f : m_new;
  // (exponentials: the bare instruction; arguments are <= 0, and results
  // below the normal range count as 0 here)
  const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
  bf16x8 ph, pl;
  float psum = 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float pe = __builtin_amdgcn_exp2f(sv[e] - m_use);
    ph[e] = f2bf(pe);
    pl[e] = f2bf(pe - bf2f(ph[e]));
    psum += pe;
  }
  psum = col4_sum(psum);
  // The running output is rescaled only when some lane needs it: a lane whose
  // maximum did not move (alpha 1) or that has accumulated nothing yet (its
  // output is 0) is unchanged by it, so skipping is exact.
  const bool rescale = !__all(alpha == 1.0f || l_run == 0.0f);  // (wave-uniform)
  l_run = l_run * alpha + psum;
  m_run = m_new;
  if (rescale) {
#pragma unroll
    for (int db = 0; db < NB; ++db) oacc[db] = oacc[db] * alpha;
  }
  if (key0 + 32 > lim) {  // (wave-uniform) the last step of the key range
    const int valid = lim - (key0 + 8 * g);
#pragma unroll
    for (int db = 0; db < NB; ++db) {
      bf16x8 a = R.f[2 * NS + db];
#pragma unroll
      for (int e = 0; e < 8; ++e) a[e] = e < valid ? a[e] : (bf16)0.0f;
      oacc[db] = mfma16x16x32(a, ph, oacc[db]);
      oacc[db] = mfma16x16x32(a, pl, oacc[db]);
    }
  } else {
#pragma unroll
    for (int db = 0; db < NB; ++db) {
      oacc[db] = mfma16x16x32(R.f[2 * NS + db], ph, oacc[db]);
      oacc[db] = mfma16x16x32(R.f[2 * NS + db], pl, oacc[db]);
    }
  }
}

// Tree attention phase.  Unit (head, 16-row block, key split) per workgroup;
// the KS splits of a (head, row block) take contiguous runs of the key range's
// 32-key steps (the prefix, then the tree's n_t slots), the last one ending
// with the tree.  Node i attends to the prefix and to the cache slots of its
// ancestors-or-self (a 128-bit set per node).  The four waves take a unit's
// steps in turn; the steps that hold prefix keys only (this pass does not
// write the prefix) are fetched before the phase's barrier, a wave's first
// two into registers and the next into its share of the LDS, so after the
// barrier only the queries and the tree's keys (written by the QKV phase) are
// waited for.  The waves' partial results are merged in LDS, in wave order;
// with KS > 1 the prefix-only splits store their partial results and the
// tree's split merges them with its own, in split order.  MB: 16-row blocks
// of the pass.
template <int MB, int DH>
__device__ __attribute__((noinline, not_tail_called)) bool attn_phase(KParams& pin, int layer, int phase, char* lds,
                                                                     int* lds_flag) {
  KParams& p = uniform_params(pin);
  const Sync sy = make_sync(p, lds_flag);
  layer = wave_uniform(layer);
  phase = wave_uniform(phase);
  using PF = AttnPrefetch<DH>;
  constexpr int KSTEPS = DH / 32, DB = DH / 16;
  const int KS = wave_uniform(p.attn_splits);
  const int rbn = wave_uniform((p.n + 15) / 16);  // row blocks holding nodes
  const int units = wave_uniform(p.H) * rbn * KS;
  const int wave = wave_index(), lane = threadIdx.x & 63, li = lane & 15, g = lane >> 4;
  const int P = wave_uniform(p.prefix_len), n = wave_uniform(p.n);
  const int nt = wave_uniform(p.nt), m0 = wave_uniform(p.m0);  // the tree's nodes; node of row 0
  const int cap = wave_uniform(p.cap);
  const int limit = P + nt;                 // keys: prefix [0, P), then the tree's slots [P, P + nt)
  const int nsteps = (limit + 31) / 32;     // 32-key steps of the key range
  const size_t kv_layer = (size_t)p.H * cap * DH;
  const bf16* kcl = p.k_cache + (size_t)layer * kv_layer;
  const bf16* vtl = p.v_cache + (size_t)layer * kv_layer;
  const bf16* qb = p.q + (size_t)layer * p.Mp * p.d;
  bf16* obase = p.o + (size_t)layer * p.Mp * p.d;
  const bf16x8* zero = (const bf16x8*)p.zero + lane;
  // step range [s_lo, s_hi) of split ks; keys of the split end at lim.  When
  // the steps do not divide evenly the first splits take the extra ones: the
  // last split holds the tree's keys, whose step is only read after the
  // barrier, and is the one the merge most often waits for.
  auto split_steps = [&](int ks, int& s_lo, int& s_hi, int& lim) {
    s_lo = (ks * nsteps + KS - 1) / KS;
    s_hi = ((ks + 1) * nsteps + KS - 1) / KS;
    lim = 32 * s_hi < limit ? 32 * s_hi : limit;
  };
  // A step can be fetched before the barrier when no cache line it touches
  // holds a tree slot: the QKV phase writes the tree's slots (with stores that
  // go to memory), and a line read into this XCD's L2 before then would stay
  // stale.  K rows are whole lines per key; a V^T row holds 64 slots per
  // 128-byte line (rows start on lines: the capacity is a multiple of 64), so
  // the step must end at or before the last 64-slot boundary of the prefix.
  const int P_lines = P & ~63;
  auto early = [&](int j) { return 32 * j + 32 <= P_lines; };

  // Attention units are dealt out so that each head's units (its row blocks
  // and key splits, which read the same keys and values) sit together on one
  // XCD and consecutive heads on consecutive XCDs: workgroup w (on XCD w % 8)
  // takes, in round k, the unit of head (q / R) 8 + w % 8 numbered q % R
  // within the head, q = (w + k G) / 8, R = units per head.  (With a grid
  // that is not a multiple of 8, unit i = w + k G.)  Within a head the units
  // keep their order, so a merging split's partners come earlier or in the
  // same round and every wait ends.
  const int R = rbn * KS;
  const int G = wave_uniform(p.G);
  const bool by_xcd = G % kXcds == 0;
  auto unit_of = [&](int i) {  // unit of slot i, or -1 (no unit), or -2 (past the last)
    if (!by_xcd) return i < units ? i : -2;
    const int q = i / kXcds, h = (q / R) * kXcds + i % kXcds;
    if ((q / R) * kXcds >= p.H) return -2;
    return h < p.H ? h * R + q % R : -1;
  };

  AttnStep<DH> A, B;
  const int wg = blockIdx.x;
  const bool prefetch = p.attn_prefetch != 0;
  {
    const int u = prefetch ? unit_of(wg) : -1;
    if (u >= 0) {
      const int h = u / R, ks = u % KS;
      const bf16* kc = kcl + (size_t)h * cap * DH;
      const bf16* vt = vtl + (size_t)h * cap * DH;
      int s_lo, s_hi, lim;
      split_steps(ks, s_lo, s_hi, lim);
      const int j0 = s_lo + wave;
      if (wave == 1) {  // wave 0's first steps, into its LDS slots
        for (int i = 0; i < PF::W0; ++i) {
          const int j = s_lo + 4 * i;
          if (j < s_hi && early(j)) attn_copy<DH>(lds + (size_t)i * PF::STEP_BYTES, kc, vt, cap, 32 * j, lim, zero);
        }
      }
      if (wave != 0) {
        if (j0 < s_hi && early(j0)) attn_load<DH>(A, kc, vt, cap, 32 * j0, lim, zero);
        if (j0 + 4 < s_hi && early(j0 + 4)) attn_load<DH>(B, kc, vt, cap, 32 * (j0 + 4), lim, zero);
        for (int i = PF::REG; i < PF::REG + PF::lds(wave); ++i) {
          const int j = j0 + 4 * i;
          if (j < s_hi && early(j))
            attn_copy<DH>(lds + (size_t)(PF::slot0(wave) + i - PF::REG) * PF::STEP_BYTES, kc, vt, cap, 32 * j, lim,
                          zero);
        }
      }
    }
  }
  trace_mark(sy, phase, 0);
  if (!grid_wait(sy, phase, p.G)) return false;
  trace_mark(sy, phase, 1);
  // The prefetched steps have landed (each wave's own loads and copies), and
  // wave 1's copies for wave 0 are visible to it.
  __builtin_amdgcn_s_waitcnt(0);
  lds_barrier();

  for (int i_slot = wg, round = 0;; i_slot += G, ++round) {
    const int u = unit_of(i_slot);
    if (u == -2) break;
    if (u < 0) continue;
    const bool first_unit = round == 0 && prefetch;
    const int h = u / R, rb = (u / KS) % rbn, ks = u % KS;
    const bf16* kc = kcl + (size_t)h * cap * DH;
    const bf16* vt = vtl + (size_t)h * cap * DH;
    int s_lo, s_hi, lim;
    split_steps(ks, s_lo, s_hi, lim);
    const int j0 = s_lo + wave;
    const int cnt = j0 < s_hi ? (s_hi - j0 + 3) / 4 : 0;  // this wave's steps: j0 + 4 i, i < cnt
    // Query fragments (B operand of S^T = K q^T): lane holds row 16 rb + li,
    // dims 32 s + 8 g + e (queries were rotated by the QKV phase).
    bf16x8 qf[KSTEPS];
    uint32_t anc[4];
    const int row = 16 * rb + li;
    {
      const bf16* qrow = qb + (size_t)row * p.d + h * DH;
#pragma unroll
      for (int s2 = 0; s2 < KSTEPS; ++s2) qf[s2] = ldg((const bf16x8*)(qrow + 32 * s2 + 8 * g));
      const int node = m0 + row < kMaxNodes ? m0 + row : kMaxNodes - 1;  // (rows past n: any node)
      const uint32_t* ap = (const uint32_t*)(p.tree + 512) + node * 4;
#pragma unroll
      for (int w = 0; w < 4; ++w) anc[w] = ldg(ap + w);
    }
    // Where step i of this wave is: in a register buffer (fetched before the
    // barrier), in an LDS slot (copied before the barrier), or still in memory.
    const int nreg = first_unit ? PF::reg(wave) : 0, nlds = first_unit ? PF::lds(wave) : 0;
    auto fetch = [&](AttnStep<DH>& R_, int i) {
      const int j = j0 + 4 * i;
      if (i >= nreg && i < nreg + nlds && i < cnt && early(j))
        attn_from_lds<DH>(R_, lds + (size_t)(PF::slot0(wave) + i - nreg) * PF::STEP_BYTES);
      else
        attn_load<DH>(R_, kc, vt, cap, 32 * j, lim, zero);
    };
    if (!(nreg > 0 && cnt > 0 && early(j0))) fetch(A, 0);
    if (!(nreg > 1 && cnt > 1 && early(j0 + 4))) fetch(B, 1);
    trace_mark(sy, phase, 3);
    float m_run = -INFINITY, l_run = 0.0f;
    f32x4 oacc[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[db] = f32x4{0.f, 0.f, 0.f, 0.f};
    // step i + 2 refills the buffer step i leaves
    for (int i = 0; i < cnt; i += 2) {
      attn_compute<DH>(A, qf, anc, 32 * (j0 + 4 * i), P, lim, p.scale_log2, m_run, l_run, oacc);
      if (i + 2 < cnt) fetch(A, i + 2);
      if (i + 1 >= cnt) break;
      attn_compute<DH>(B, qf, anc, 32 * (j0 + 4 * (i + 1)), P, lim, p.scale_log2, m_run, l_run, oacc);
      if (i + 3 < cnt) fetch(B, i + 3);
    }
    trace_mark(sy, phase, 4);
    // The four waves' partial results -> LDS (the prefetch slots are spent),
    // merged in wave order: o = sum_w exp2(m_w - M) o_w / sum_w exp2(m_w - M) l_w
    // (unnormalised when the key splits still have to be merged).
    lds_barrier();
    float* mlm = reinterpret_cast<float*>(lds);  // [4][16][2]
    float* om = mlm + kWaves * 16 * 2;          // [4][16][DH]
    if (g == 0) {
      lds_st<float>(&mlm[(wave * 16 + li) * 2], m_run);
      lds_st<float>(&mlm[(wave * 16 + li) * 2 + 1], l_run);
    }
#pragma unroll
    for (int db = 0; db < DB; ++db) lds_st<f32x4>(&om[(size_t)(wave * 16 + li) * DH + 16 * db + 4 * g], oacc[db]);
    lds_barrier();
    const size_t rbi = (size_t)h * MB + rb;  // (head, row block) slot
    // This thread's items of the unit's result: row it / (Dh/2), columns
    // dd, dd + 1 (it = thread + k * threads).
    constexpr int NIT = 16 * (DH / 2) / kThreads;
    static_assert(NIT * kThreads == 16 * (DH / 2), "items per thread");
    float uM[NIT], uL[NIT], u0[NIT], u1[NIT];
#pragma unroll
    for (int k = 0; k < NIT; ++k) {
      const int it = threadIdx.x + k * kThreads;
      const int i = it / (DH / 2), dd = 2 * (it % (DH / 2));
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) M = fmaxf(M, lds_ld<float>(&mlm[(w * 16 + i) * 2]));
      float L = 0.0f, o0 = 0.0f, o1 = 0.0f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float m = lds_ld<float>(&mlm[(w * 16 + i) * 2]);
        const float wt = m == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(m - M);
        L += lds_ld<float>(&mlm[(w * 16 + i) * 2 + 1]) * wt;
        const float2 ov = lds_ld<float2>(&om[(size_t)(w * 16 + i) * DH + dd]);
        o0 += ov.x * wt;
        o1 += ov.y * wt;
      }
      uM[k] = M;
      uL[k] = L;
      u0[k] = o0;
      u1[k] = o1;
    }
    // With key splits, every split stores its partial result and counts its
    // arrival on the (head, row block) counter; the last to arrive merges all
    // of them (no split waits for another), in split order whichever split
    // that is, so the result is bit-reproducible.
    bool merge = true;
    if (KS > 1) {
#pragma unroll
      for (int k = 0; k < NIT; ++k) {
        const int it = threadIdx.x + k * kThreads;
        const int i = it / (DH / 2), dd = 2 * (it % (DH / 2));
        const size_t sl = rbi * KS + ks;
        st_coherent2(&p.attn_o[(sl * 16 + i) * DH + dd], u0[k], u1[k]);
        if (dd == 0) st_coherent2(&p.attn_ml[(sl * 16 + i) * 2], uM[k], uL[k]);
      }
      merge = arrive_last(&p.head_cnt[rbi], KS, lds_flag);
      if (merge) trace_mark(sy, phase, 6);
    }
    if (merge) {
      constexpr int SO = kAttnMaxSplits;
      float2 ml[NIT][SO], ov[NIT][SO];
#pragma unroll
      for (int k = 0; k < NIT; ++k) {
        const int it = threadIdx.x + k * kThreads;
        const int i = it / (DH / 2), dd = 2 * (it % (DH / 2));
#pragma unroll
        for (int s2 = 0; s2 < SO; ++s2) {
          const bool other = s2 < KS && s2 != ks;
          const size_t sl = rbi * KS + (other ? s2 : 0);
          ml[k][s2] = other ? ld_coherent2(&p.attn_ml[(sl * 16 + i) * 2])
                            : (s2 == ks ? make_float2(uM[k], uL[k]) : make_float2(-INFINITY, 0.0f));
          ov[k][s2] = other ? ld_coherent2(&p.attn_o[(sl * 16 + i) * DH + dd])
                            : (s2 == ks ? make_float2(u0[k], u1[k]) : make_float2(0.0f, 0.0f));
        }
      }
#pragma unroll
      for (int k = 0; k < NIT; ++k) {
        const int it = threadIdx.x + k * kThreads;
        const int i = it / (DH / 2), dd = 2 * (it % (DH / 2));
        const int r = 16 * rb + i;
        float M = -INFINITY;
#pragma unroll
        for (int s2 = 0; s2 < SO; ++s2) M = fmaxf(M, ml[k][s2].x);
        float L = 0.0f, o0 = 0.0f, o1 = 0.0f;
#pragma unroll
        for (int s2 = 0; s2 < SO; ++s2) {
          const float wt = ml[k][s2].x == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(ml[k][s2].x - M);
          L += ml[k][s2].y * wt;
          o0 += ov[k][s2].x * wt;
          o1 += ov[k][s2].y * wt;
        }
        const float inv = 1.0f / L;
        if (r < n) st_coherent_bf2(obase + frag_off(r, h * DH + dd, MB), o0 * inv, o1 * inv);
        if (k == 0) trace_mark(sy, phase, 7);
      }
    }
    trace_mark(sy, phase, 5);
    lds_barrier();
  }
  return true;
}

// ------------------------------------------------------------------ embed

// Tree preparation (every node's depth, position prefix_len + depth, and
// ancestor-or-self set: its row of the tree masking table) and the residual
// stream's first version: the nodes' embedding rows, bf16(x * g) for the
// first layer's norm, and the sums of squares of every 16 columns.
template <int MB>
__device__ __forceinline__ void embed_phase(KParams& p, const TreeArgs& tree, int* par_s) {
  const bf16* E = (const bf16*)(p.packed + p.o_embed);
  if (blockIdx.x == 0) {
    if (threadIdx.x < 128) par_s[threadIdx.x] = threadIdx.x < p.nt ? tree.parent[threadIdx.x] : -1;
    __syncthreads();
    if (threadIdx.x < 128) {
      const int i = threadIdx.x;
      int dep = 0;
      uint32_t a[4] = {0u, 0u, 0u, 0u};
      if (i < p.nt) {
        for (int j = i; j >= 0; j = par_s[j]) {
          a[j >> 5] |= 1u << (j & 31);
          ++dep;
        }
        --dep;
      }
      st_coherent(&p.tree[i], i < p.nt ? tree.tok[i] : 0);
      st_coherent(&p.tree[128 + i], par_s[i]);
      st_coherent(&p.tree[256 + i], dep);
      st_coherent(&p.tree[384 + i], p.prefix_len + dep);
#pragma unroll
      for (int w = 0; w < 4; ++w) st_coherent(&p.tree[512 + i * 4 + w], (int)a[w]);
    }
  }
  const int lane = threadIdx.x & 63;
  for (int m = blockIdx.x; m < p.n; m += p.G) {
    // rotary table row m (node m0 + m): (cos, sin) of its position times
    // theta^(-2j/Dh), j < Dh/2
    if (threadIdx.x < p.Dh / 2) {
      int dep = 0;
      for (int j = tree.parent[p.m0 + m]; j >= 0; j = tree.parent[j]) ++dep;
      const int jj = threadIdx.x;
      float sn, cs;
      sincosf((float)(p.prefix_len + dep) * rope_inv_freq(jj, p.Dh, p.log2_theta), &sn, &cs);
      st_coherent2(p.rope + ((size_t)m * (p.Dh / 2) + jj) * 2, cs, sn);
    }
  }
  // The stream's first version, dealt out over every workgroup by element
  // (node m, column c) in row-major order -- 16 consecutive lanes hold one
  // 16-column block of one row -- with each thread's loads all issued before
  // its stores.
  const bf16* g0 = (const bf16*)(p.packed + p.layer0 + p.o_attn_norm);
  const int total = p.n * p.d, stride = p.G * kThreads;
  constexpr int PER = 4;
  for (int base = blockIdx.x * kThreads; base < total; base += PER * stride) {
    float v[PER], g[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = base + k * stride + threadIdx.x;
      const int m = e < total ? e / p.d : 0, c = e < total ? e % p.d : 0;
      v[k] = e < total ? bf2f(ldg(E + (size_t)tree.tok[p.m0 + m] * p.d + c)) : 0.0f;
      g[k] = e < total ? bf2f(ldg(g0 + c)) : 0.0f;
    }
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = base + k * stride + threadIdx.x;
      const int m = e / p.d, c = e % p.d;
      const float xg = v[k] * g[k];
      const float xg1 = dpp_f<kDppRowShl1>(xg);
      const float sq = row16_sum(v[k] * v[k]);  // sum of squares over the 16-column block
      if (e < total) {
        st_coherent(&p.x[(size_t)m * p.d + c], v[k]);
        if ((c & 1) == 0) st_coherent_bf2(p.xg + frag_off(m, c, MB), xg, xg1);
        if ((lane & 15) == 0) st_coherent(&p.ssq[(size_t)(c / kNB) * p.Mp + m], sq);
      }
    }
  }
}

// ------------------------------------------------------------------ kernel

// Dynamic LDS: the GEMM tiles' region (all LDS but the static part), which
// the attention reuses for its prefetched steps and its merge.
template <int DH>
constexpr size_t dyn_lds_bytes() {
  static_assert(AttnPrefetch<DH>::W0 >= 1 && AttnPrefetch<DH>::W23 >= 1 &&
                    (size_t)(AttnPrefetch<DH>::W0 + 2 * AttnPrefetch<DH>::W23) * AttnPrefetch<DH>::STEP_BYTES <=
                        kGemmLdsBytes,
                "attention prefetch slots");
  static_assert((size_t)kWaves * 16 * (DH + 2) * 4 <= kGemmLdsBytes, "attention merge");
  return kGemmLdsBytes;
}

// ------------------------------------------------------------------ final norm

// The final RMSNorm, rounded where the model rounds it: xnf = bf16(x rstd g)
// of the last residual version, in fragment order, the LM head's input.  (A
// layer's norms round bf16(x g) instead and scale the product's rows, which
// needs no phase of its own; for the logits one phase per pass keeps the
// model's rounding point.)  Workgroup w takes the 16-column blocks
// [w d/16 / G, (w + 1) d/16 / G).
template <int MB>
__device__ __attribute__((noinline, not_tail_called)) bool final_norm_phase(KParams& pin, int phase, GemmLds& gl,
                                                                           int* lds_flag) {
  KParams& p = uniform_params(pin);
  phase = wave_uniform(phase);
  const Sync sy = make_sync(p, lds_flag);
  trace_mark(sy, phase, 0);
  if (!grid_wait(sy, phase, p.G)) return false;
  trace_mark(sy, phase, 1);
  constexpr int ROWS = 16 * MB;
  row_rstd<MB>(p, p.ssq + (size_t)(2 * p.L) * p.d_nb * p.Mp, gl);
  const float* x = p.x + (size_t)(2 * p.L) * p.Mp * p.d;
  const bf16* g = (const bf16*)(p.packed + p.o_final_norm);
  const int vw = virtual_wg(p.G);
  const int lo = wave_uniform((int)((long)vw * p.d_nb / p.G));
  const int hi = wave_uniform((int)((long)(vw + 1) * p.d_nb / p.G));
  for (int e = threadIdx.x; e < (hi - lo) * ROWS * (kNB / 2); e += kThreads) {
    const int pr = e % (kNB / 2), r = (e / (kNB / 2)) % ROWS, b = lo + e / ((kNB / 2) * ROWS);
    const int c = kNB * b + 2 * pr;
    if (r < p.n) {
      const float2 xv = ldg((const float2*)(x + (size_t)r * p.d + c));
      const float s = gl.rstd[r];
      st_coherent_bf2(p.xnf + frag_off(r, c, MB), xv.x * s * bf2f(g[c]), xv.y * s * bf2f(g[c + 1]));
    }
  }
  trace_mark(sy, phase, 5);
  return true;
}

// WIDE: gate/up tiles of up to 9 blocks (a separate kernel, so that the
// other kernels' code is unchanged by it).
template <int MB, int DH, bool WIDE = false>
__global__ __launch_bounds__(kThreads, 1) void pass_kernel(const PassParams p_arg, const TreeArgs tree) {
  extern __shared__ __attribute__((aligned(1024))) char lds_raw[];
  __shared__ GemmLds gl;
  __shared__ int par_s[128];
  __shared__ int flag;
  // The parameter block is the first kernel argument: read it in place.
  KParams& p = *(KParams*)__builtin_amdgcn_kernarg_segment_ptr();
  if (p.magic != kPassMagic || p.G != p_arg.G || p.n != p_arg.n || p.Mp != 16 * MB) {
    if (threadIdx.x == 0 && blockIdx.x == 0) stg(p_arg.status, 3);
    return;  // (uniform over the grid: no workgroup reaches a barrier)
  }
  const Sync sy = make_sync(p, &flag);
  int phase = 0;
  bool ok = true;

  embed_phase<MB>(p, tree, par_s);
  grid_arrive(sy, phase);
  ++phase;
  // The QKV phases load the rotary table before they wait at their barrier
  // (it is written long before, except for the first layer's): one more
  // barrier publishes it.
  ok = grid_wait(sy, phase, p.G);
  grid_arrive(sy, phase);
  ++phase;

  for (int l = 0; l < p.L && ok; ++l) {
    ok = gemm_phase<MB, EPI_QKV>(p, STEP_QKV, l, phase, lds_raw, gl, &flag);
    if (!ok) break;
    grid_arrive(sy, phase++);
    ok = attn_phase<MB, DH>(p, l, phase, lds_raw, &flag);
    if (!ok) break;
    grid_arrive(sy, phase++);
    ok = p.step[STEP_O].split > 1 ? split_phase<MB, EPI_RESID>(p, STEP_O, l, phase, lds_raw, gl, &flag)
                                  : gemm_phase<MB, EPI_RESID>(p, STEP_O, l, phase, lds_raw, gl, &flag);
    if (!ok) break;
    grid_arrive(sy, phase++);
    ok = gemm_phase<MB, EPI_SWIGLU, WIDE ? 9 : 8>(p, STEP_GATE_UP, l, phase, lds_raw, gl, &flag);
    if (!ok) break;
    grid_arrive(sy, phase++);
    ok = p.step[STEP_DOWN].split > 1
             ? split_phase<MB, EPI_RESID>(p, STEP_DOWN, l, phase, lds_raw, gl, &flag)
             : gemm_phase<MB, EPI_RESID>(p, STEP_DOWN, l, phase, lds_raw, gl, &flag);
    if (!ok) break;
    grid_arrive(sy, phase++);
  }
  if (ok) ok = final_norm_phase<MB>(p, phase, gl, &flag);
  if (ok) {  // LM head + argmax + accept walk
    grid_arrive(sy, phase++);
    if (gemm_phase<MB, EPI_LOGITS>(p, STEP_LM, 0, phase, lds_raw, gl, &flag)) trace_mark(sy, phase, 2);
  }
  // Leave the pass: the last workgroup out resets the barrier and split-K
  // group counters.
  if (arrive_last(p.exit_cnt, p.G, &flag)) {
    if (threadIdx.x < kBarSlots) st_coherent(p.bar + threadIdx.x * kBarStride, 0);
    if (p.step[STEP_O].split > 1 || p.step[STEP_DOWN].split > 1)
      for (int i = threadIdx.x; i < p.G / 2; i += kThreads) {
        st_coherent(p.grp_cnt + i, 0);
        st_coherent(p.grp_cnt + kPassMaxGrid / 2 + i, 0);
      }
  }
}

template <int MB, int DH, bool WIDE>
hipError_t launch_pass_mb(KParams& p, const TreeArgs& tree, hipStream_t st) {
  static bool attr_set = false;  // per process; the attribute is per function
  const void* fn = (const void*)pass_kernel<MB, DH, WIDE>;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn_lds_bytes<DH>());
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  void* args[] = {(void*)&p, (void*)&tree};
  return hipLaunchCooperativeKernel(fn, dim3(p.G), dim3(kThreads), args, (unsigned)dyn_lds_bytes<DH>(), st);
}

template <int MB, int DH, bool WIDE>
int occupancy_mb() {
  const void* fn = (const void*)pass_kernel<MB, DH, WIDE>;
  if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn_lds_bytes<DH>()) != hipSuccess)
    return 0;
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, fn, kThreads, dyn_lds_bytes<DH>()) != hipSuccess)
    return 0;
  return blocks;
}

}  // namespace

hipError_t launch_pass(int mb16, KParams& p, const TreeArgs& tree, hipStream_t st) {
  const bool wide = p.step[STEP_GATE_UP].wide != 0;  // (set for 16- and 32-row passes only)
#define LLMCAD_PASS_CASE(M, W)                                              \
  case M:                                                                   \
    return p.Dh == 128 ? launch_pass_mb<M, 128, W>(p, tree, st)             \
                       : launch_pass_mb<M, 64, W>(p, tree, st);
  if (!wide) {
    switch (mb16) {
      LLMCAD_PASS_CASE(1, false)
      LLMCAD_PASS_CASE(2, false)
      LLMCAD_PASS_CASE(4, false)
      LLMCAD_PASS_CASE(8, false)
      default:
        return hipErrorInvalidValue;
    }
  }
  switch (mb16) {
    LLMCAD_PASS_CASE(1, true)
    LLMCAD_PASS_CASE(2, true)
    default:
      return hipErrorInvalidValue;
  }
#undef LLMCAD_PASS_CASE
}

int pass_occupancy(int mb16, int dh, bool wide) {
#define LLMCAD_OCC_CASE(M, W) \
  case M:                     \
    return dh == 128 ? occupancy_mb<M, 128, W>() : occupancy_mb<M, 64, W>();
  if (!wide) {
    switch (mb16) {
      LLMCAD_OCC_CASE(1, false)
      LLMCAD_OCC_CASE(2, false)
      LLMCAD_OCC_CASE(4, false)
      LLMCAD_OCC_CASE(8, false)
      default:
        return 0;
    }
  }
  switch (mb16) {
    LLMCAD_OCC_CASE(1, true)
    LLMCAD_OCC_CASE(2, true)
    default:
      return 0;
  }
#undef LLMCAD_OCC_CASE
}

size_t pass_lds_bytes(int mb16, int dh) {
  (void)mb16;
  return dh == 128 ? dyn_lds_bytes<128>() : dyn_lds_bytes<64>();
}

}  // namespace llmcad
