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
// Phases: embed + tree prep; per layer QKV projection (RMSNorm applied to
// the staged activations; rotary embedding and K/V cache write in the
// epilogue) -> tree attention (ancestor mask) -> O projection (+residual) ->
// gate/up (RMSNorm; SwiGLU epilogue) -> down projection (+residual); then
// final RMSNorm + LM head + argmax, and the accept walk in the workgroup that
// completes the argmax.
//
// GEMM phases (activations X [Mp rows x K], packed weights W [N x K]): the
// host cuts every step into tiles (GemmPlan): a tile is a group of up to 16
// consecutive 32-column n-blocks times a slice of the k-steps.  A tile's
// activation slice is copied once into LDS with direct global->LDS loads, in
// exactly the lane order of the 32x32x16 MFMA A operand, while the weights
// stream from HBM through a register pipeline (non-temporal loads); the
// activations are never re-read from L2 per n-block.  The four waves take
// interleaved k-steps and their partial tiles are added in LDS in wave
// order.  When a group's k-steps are split over S tiles, each tile stores its
// partial sum and the workgroup that completes the group last adds the S
// partials in slice order (bit-reproducible) and runs the epilogue.
//
// Coherence without cache maintenance: every buffer handed from one phase to
// the next is written once per pass at its own address with device-coherent
// stores and read after the barrier with ordinary loads, so no L2 can hold an
// older copy; buffers reused within a pass (partials) are read with
// device-coherent loads.  Barriers and per-head joins are counters polled
// with bounded spins: a wait that exceeds its bound records an error status
// and the workgroup leaves the pass, so no wave can hang.
#include <math.h>

#include "device.h"
#include "kernels.h"
#include "layout.h"

namespace llmcad {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;

typedef float f32x16 __attribute__((ext_vector_type(16)));

enum Epilogue { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_LOGITS = 3 };
constexpr int kTraceWgs = 8;  // workgroups that record phase timestamps

// D = A(32x16) * B(16x32) + C on the matrix cores, bf16 inputs, fp32
// accumulate.  Lane l holds A row l % 32 and B column l % 32, k-slots
// 8 (l / 32) .. + 7 of both; D element i of lane l is row
// 8 (i / 4) + 4 (l / 32) + i % 4, column l % 32.
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ int acc_row(int i, int lane) { return 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3); }

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

// Direct global -> LDS copy of 16 bytes per lane: lane l's bytes land at
// lds + 16 l.  `lds` must be the same in every lane.
__device__ __forceinline__ void dma16(const void* src, char* lds) {
  __builtin_amdgcn_global_load_lds((const LLMCAD_GLOBAL void*)src,
                                   (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
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
  s.trace = p.trace != nullptr && (int)blockIdx.x < kTraceWgs
                ? p.trace + (size_t)blockIdx.x * (2 + 5 * p.L) * 8
                : nullptr;
  return s;
}

// Diagnostics: wall-clock (100 MHz) marks per phase: 0 = barrier wait
// entered, 1 = wait over, 2 = phase work done; GEMM phases also mark 3 =
// activations staged, 4 = weight streaming done, 5 = epilogue done, 6 =
// group hand-off done, 7 = partials added (group's last workgroup).
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

// Waits until all G workgroups have arrived `phase` times; one wave polls all
// counters.  False (to all threads) if the bounded spin ran out.  The total
// is exact only because every workgroup waits at every phase before it
// arrives again: no workgroup can then be more than one arrival ahead.
__device__ __forceinline__ bool grid_wait(const Sync& s, int phase, int G) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    const int slots = G < kBarSlots ? G : kBarSlots;
    const int per = G / kBarSlots + (lane < G % kBarSlots ? 1 : 0);
    const int want = lane < slots ? phase * (G < kBarSlots ? 1 : per) : 0;
    const int* slot = s.bar + (lane < slots ? lane : 0) * kBarStride;
    int ok = 1, spins = 0;
    while (true) {
      const int v = lane < slots ? ld_coherent(slot) : 0;
      if (__all(v >= want)) break;
      __builtin_amdgcn_s_sleep(1);
      if (++spins > s.limit) {
        if (lane == 0) st_coherent(s.status, 1);
        ok = 0;
        break;
      }
    }
    if (lane == 0) *s.lds_flag = ok;
  }
  __syncthreads();
  const bool ok = *s.lds_flag != 0;
  __syncthreads();
  return ok;
}

// Waits until *c >= target (one poller); false if the bounded spin ran out.
__device__ __forceinline__ bool wait_at_least(const Sync& s, const int* c, int target) {
  if (threadIdx.x == 0) {
    int ok = 1, spins = 0;
    while (ld_coherent(c) < target) {
      __builtin_amdgcn_s_sleep(1);
      if (++spins > s.limit) {
        st_coherent(s.status, 1);
        ok = 0;
        break;
      }
    }
    *s.lds_flag = ok;
  }
  __syncthreads();
  const bool ok = *s.lds_flag != 0;
  __syncthreads();
  return ok;
}

// ------------------------------------------------------------------ GEMM

struct GemmLds {
  float rstd[kMaxNodes];          // RMSNorm scale per row of the current tile
  float part_ss[256];             // their partial sums
  float red_v[kMaxNodes][kMaxCW]; // LM head: argmax per (row, n-block)
  int red_i[kMaxNodes][kMaxCW];
  int reach[kMaxNodes];
  int amax[kMaxNodes];
  int tok[kMaxNodes];  // accept walk: the tree, staged from the workspace
  int par[kMaxNodes];
  int dep[kMaxNodes];
  int walk_len;
};

// What one GEMM step reads and writes in a given layer.  The activations
// of every step are bf16 [Mp][lda]: the attention output, the SwiGLU
// product, or, for the steps behind an RMSNorm, bf16(x * g) of the residual
// version x with that norm's gain g; the norm's per-row scale
// 1 / sqrt(mean(x^2) + eps) is then applied to the step's output rows.
struct StepIo {
  const bf16x8* w;   // packed matrix
  int ks;            // k-steps per n-block (K / 16)
  bool norm;         // rows of the output are scaled by the norm's rstd
  const bf16* a;     // [Mp][lda]
  int lda;
  const float* ssq;  // norm: [d/32][Mp] sums of squares of the residual version
  // epilogue
  bf16* q;           // QKV: [Mp][d] queries after the rotary embedding
  bf16* kc;          // QKV: K cache of this layer [H][cap][Dh]
  bf16* vc;          // QKV: V cache of this layer [H][cap][Dh]
  const float* x_in; // RESID: [Mp][d]
  float* x_out;      // RESID: [Mp][d]
  float* ssq_out;    // RESID: [d/32][Mp]
  bf16* xg_out;      // RESID: [Mp][d] bf16(x_out * g_next)
  const bf16* g_next;  // RESID: gain of the norm that reads x_out
  bf16* h;           // SWIGLU: [Mp][Fp]
};

__device__ __forceinline__ StepIo step_io(KParams& p, int step, int l) {
  const size_t xsz = (size_t)p.Mp * p.d, ssz = (size_t)p.d_nb * p.Mp;
  const char* lw = p.packed + p.layer0 + (long long)l * p.layer_bytes;
  const StepPlan& sp = p.step[step];
  StepIo io{};
  io.w = (const bf16x8*)((sp.layer_rel ? lw : p.packed) + sp.w_off);
  io.ks = sp.ksteps;
  switch (step) {
    case STEP_QKV:
      io.norm = true;
      io.a = p.xg + (size_t)(2 * l) * xsz;
      io.lda = p.d;
      io.ssq = p.ssq + (size_t)(2 * l) * ssz;
      io.q = p.q + (size_t)l * p.Mp * p.d;
      io.kc = p.k_cache + (size_t)l * p.H * p.cap * p.Dh;
      io.vc = p.v_cache + (size_t)l * p.H * p.cap * p.Dh;
      break;
    case STEP_O:
      io.norm = false;
      io.a = p.o + (size_t)l * p.Mp * p.d;
      io.lda = p.d;
      io.x_in = p.x + (size_t)(2 * l) * xsz;
      io.x_out = p.x + (size_t)(2 * l + 1) * xsz;
      io.ssq_out = p.ssq + (size_t)(2 * l + 1) * ssz;
      io.xg_out = p.xg + (size_t)(2 * l + 1) * xsz;
      io.g_next = (const bf16*)(lw + p.o_ffn_norm);
      break;
    case STEP_GATE_UP:
      io.norm = true;
      io.a = p.xg + (size_t)(2 * l + 1) * xsz;
      io.lda = p.d;
      io.ssq = p.ssq + (size_t)(2 * l + 1) * ssz;
      io.h = p.h + (size_t)l * p.Mp * p.Fp;
      break;
    case STEP_DOWN:
      io.norm = false;
      io.a = p.h + (size_t)l * p.Mp * p.Fp;
      io.lda = p.Fp;
      io.x_in = p.x + (size_t)(2 * l + 1) * xsz;
      io.x_out = p.x + (size_t)(2 * l + 2) * xsz;
      io.ssq_out = p.ssq + (size_t)(2 * l + 2) * ssz;
      io.xg_out = p.xg + (size_t)(2 * l + 2) * xsz;
      io.g_next = l + 1 < p.L ? (const bf16*)(lw + p.layer_bytes + p.o_attn_norm)
                              : (const bf16*)(p.packed + p.o_final_norm);
      break;
    default:  // STEP_LM
      io.norm = true;
      io.a = p.xg + (size_t)(2 * p.L) * xsz;
      io.lda = p.d;
      io.ssq = p.ssq + (size_t)(2 * p.L) * ssz;
      break;
  }
  return io;
}

// Copies the tile's activation slice (k-steps [k0, k0 + kt), all Mp rows)
// into LDS in MFMA A-operand lane order: unit (kk, mb) = 1 KiB at
// (kk MB + mb) KiB, lane l's 16 bytes = row 32 mb + l % 32, inputs
// 16 (k0 + kk) + 8 (l / 32) .. + 7.  Rows >= n read zeros.  Waves take units
// in turn; the caller waits for the loads.
template <int MB>
__device__ __forceinline__ void stage_activations(KParams& p, const StepIo& io, int k0, int kt, char* A) {
  const int wave = wave_index(), lane = threadIdx.x & 63;
  const int lrow = lane & 31, khalf = lane >> 5;
  const char* zero = p.zero + lane * 16;
  const int units = kt * MB;
  for (int u = wave; u < units; u += kWaves) {
    const int kk = u / MB, mb = u % MB;
    const int r = 32 * mb + lrow;
    const void* src = r < p.n ? (const void*)(io.a + (size_t)r * io.lda + 16 * (k0 + kk) + 8 * khalf)
                              : (const void*)zero;
    dma16(src, A + (size_t)u * 1024);
  }
}

// RMSNorm scales of rows [0, Mp): 1 / sqrt(mean of squares + eps) from the
// per-n-block sums of squares the producing phase wrote (added in n-block
// order); 0 for rows >= n.  Loads are issued here, the sums are formed by
// finish_row_scales after the caller's wait.
template <int MB>
struct SsqLoads {
  static constexpr int ROWS = 32 * MB, CHK = 256 / ROWS, PER = 16;
  float v[PER];
};
template <int MB>
__device__ __forceinline__ void row_scale_loads(KParams& p, const StepIo& io, SsqLoads<MB>& L, int pass) {
  constexpr int ROWS = 32 * MB, CHK = 256 / ROWS, PER = SsqLoads<MB>::PER;
  const int r = threadIdx.x % ROWS, ch = threadIdx.x / ROWS;
  const int dn = p.d_nb;
  const int t0 = ch * dn / CHK, t1 = (ch + 1) * dn / CHK;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int t = t0 + pass * PER + i;
    L.v[i] = (r < p.n && t < t1) ? ldg(io.ssq + (size_t)t * p.Mp + r) : 0.0f;
  }
}
template <int MB>
__device__ __forceinline__ void row_scales(KParams& p, const StepIo& io, GemmLds& gl) {
  constexpr int ROWS = 32 * MB, CHK = 256 / ROWS, PER = SsqLoads<MB>::PER;
  const int r = threadIdx.x % ROWS, ch = threadIdx.x / ROWS;
  const int dn = p.d_nb;
  const int len = (ch + 1) * dn / CHK - ch * dn / CHK;
  float ss = 0.0f;
  for (int pass = 0; pass * PER < len; ++pass) {
    SsqLoads<MB> L;
    row_scale_loads<MB>(p, io, L, pass);
#pragma unroll
    for (int i = 0; i < PER; ++i) ss += L.v[i];
  }
  gl.part_ss[ch * ROWS + r] = ss;
  __syncthreads();
  if (threadIdx.x < ROWS) {
    float t = 0.0f;
    for (int c = 0; c < CHK; ++c) t += gl.part_ss[c * ROWS + threadIdx.x];
    gl.rstd[threadIdx.x] = threadIdx.x < p.n ? 1.0f / sqrtf(t * p.inv_d + p.eps) : 0.0f;
  }
  __syncthreads();
}

// Weight stages per wave: about 160 VGPRs, 2 to 16 k-steps; one stage for
// the widest tiles, whose accumulators fill the AGPRs.
template <int CW>
constexpr int tile_depth() {
  constexpr int d = 40 / CW;
  return CW >= 12 ? 1 : (d < 2 ? 2 : (d > 16 ? 16 : d));
}

// One tile: n-blocks [nb0, nb0 + CW) x k-steps [k0, k1) of a step.  Issues
// the first weight stages, then (wait_phase >= 0) waits at the grid barrier
// for the step's inputs, stages the activations into LDS, streams the
// weights and leaves the tile's sum in LDS at T = A:
// fp32 [CW][MB][64 lanes][16] (MFMA accumulator order).  False if a wait
// ran out.
template <int MB, int CW>
__device__ __attribute__((noinline, not_tail_called)) bool tile_compute(KParams& pin, int step, int layer,
                                                                       int nb0, int k0, int k1,
                                                                       int wait_phase, char* A,
                                                                       GemmLds& gl, int* lds_flag) {
  KParams& p = uniform_params(pin);
  step = wave_uniform(step);
  layer = wave_uniform(layer);
  nb0 = wave_uniform(nb0);
  k0 = wave_uniform(k0);
  k1 = wave_uniform(k1);
  wait_phase = wave_uniform(wait_phase);
  const StepIo io = step_io(p, step, layer);
  const int wave = wave_index(), lane = threadIdx.x & 63;
  const int kt = k1 - k0;
  const int ns = wave_uniform(wave < kt ? (kt - wave + kWaves - 1) / kWaves : 0);
  constexpr int D = tile_depth<CW>();
  // this wave's k-steps: k0 + wave + 4 i
  const bf16x8* wt = io.w + ((size_t)nb0 * io.ks + k0 + wave) * 64 + lane;
  const size_t cstride = (size_t)io.ks * 64;
  bf16x8 bw[D][CW];
  auto load_stage = [&](int slot, int i) {
#pragma unroll
    for (int c = 0; c < CW; ++c) bw[slot][c] = ldg_nt(wt + c * cstride + (size_t)(kWaves * i) * 64);
  };
  if (ns > 0) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      load_stage(u, u < ns ? u : ns - 1);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  if (wait_phase >= 0) {
    const Sync sy = make_sync(p, lds_flag);
    trace_mark(sy, wait_phase, 0);
    if (!grid_wait(sy, wait_phase, p.G)) return false;
    trace_mark(sy, wait_phase, 1);
  }
  stage_activations<MB>(p, io, k0, kt, A);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (wait_phase >= 0 && p.trace != nullptr && (int)blockIdx.x < kTraceWgs && threadIdx.x == 0)
    stg(p.trace + (size_t)blockIdx.x * (2 + 5 * p.L) * 8 + wait_phase * 8 + 3, (long long)wall_clock64());

  f32x16 acc[MB][CW];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int c = 0; c < CW; ++c) acc[mb][c] = f32x16{};
  for (int i = 0; i < ns; i += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      __builtin_amdgcn_sched_barrier(0);
      if (i + u < ns) {
        const int kk = wave + kWaves * (i + u);
        bf16x8 a[MB];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) a[mb] = *(const bf16x8*)(A + (size_t)(kk * MB + mb) * 1024 + lane * 16);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int c = 0; c < CW; ++c) acc[mb][c] = mfma32(a[mb], bw[u][c], acc[mb][c]);
      }
      __builtin_amdgcn_sched_barrier(0);
      const int nx = i + u + D < ns ? i + u + D : ns - 1;
      load_stage(u, nx);
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  __syncthreads();  // every wave is done reading the activations
  // Wave partials -> T (the activation region), added in wave order.
  float* T = reinterpret_cast<float*>(A);
  for (int w = 0; w < kWaves; ++w) {
    if (wave == w) {
#pragma unroll
      for (int c = 0; c < CW; ++c)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          float4* dst = reinterpret_cast<float4*>(T + ((size_t)(c * MB + mb) * 64 + lane) * 16);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            float4 v = make_float4(acc[mb][c][4 * j], acc[mb][c][4 * j + 1], acc[mb][c][4 * j + 2],
                                   acc[mb][c][4 * j + 3]);
            if (w > 0) {
              const float4 o = dst[j];
              v.x += o.x;
              v.y += o.y;
              v.z += o.z;
              v.w += o.w;
            }
            dst[j] = v;
          }
        }
    }
    __syncthreads();
  }
  return true;
}

template <int MB, int CW>
__device__ __forceinline__ bool tile_dispatch(int cw, KParams& p, int step, int layer, int nb0, int k0,
                                              int k1, int wait_phase, char* A, GemmLds& gl, int* flag) {
  if constexpr (CW >= 1) {
    if (cw == CW) return tile_compute<MB, CW>(p, step, layer, nb0, k0, k1, wait_phase, A, gl, flag);
    return tile_dispatch<MB, CW - 1>(cw, p, step, layer, nb0, k0, k1, wait_phase, A, gl, flag);
  } else {
    return false;
  }
}

// Rotary embedding frequency of dim pair (j, j + Dh/2): theta^(-2j/Dh).
__device__ __forceinline__ float rope_inv_freq(int j, int Dh, float log2_theta) {
  return exp2f(-(2.0f * (float)j / (float)Dh) * log2_theta);
}

// Epilogue.  A group's output is cw n-blocks x MB row blocks, one 32x32
// accumulator tile ("unit") each, unit u = c MB + mb, held in T (fp32
// [cw][MB][64 lanes][16], MFMA accumulator order).  A workgroup finishes
// units [u_lo, u_hi): its waves take them in turn, kEpiBatch per wave at a
// time, and write the step's outputs with device-coherent stores.  The
// inputs a batch reads from memory (the residual stream, the rotary table)
// are loaded first, all at once (EpiPre), so that a batch costs one round
// trip; the first batch's are issued before the group's partials are read.
constexpr int kEpiBatch = 2;

template <int EPI>
struct EpiPre {
  static constexpr int U = (EPI == EPI_RESID || EPI == EPI_QKV) ? kEpiBatch : 1;
  float a[U][16];                       // RESID: x_in; QKV: cos
  float b[EPI == EPI_QKV ? U : 1][16];  // QKV: sin
  float g[EPI == EPI_RESID ? U : 1];    // RESID: gain of the next norm at this lane's column
};

template <int MB, int EPI>
__device__ __forceinline__ void epilogue_preload(KParams& p, const StepIo& io, int nb0, int u_lo, int u_hi, int ub,
                                                 EpiPre<EPI>& pre) {
  if constexpr (EPI == EPI_RESID || EPI == EPI_QKV) {
    const int wave = wave_index(), lane = threadIdx.x & 63;
    const int j = lane & 31;
#pragma unroll
    for (int uu = 0; uu < kEpiBatch; ++uu) {
      const int unit = u_lo + wave + kWaves * (ub + uu);
      if (unit >= u_hi) break;
      const int c = unit / MB, mb = unit % MB;
      const int nb = nb0 + c;
      if constexpr (EPI == EPI_RESID) {
        const int col = kNB * nb + j;
        pre.g[uu] = bf2f(ldg(io.g_next + col));
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = 32 * mb + acc_row(i, lane);
          pre.a[uu][i] = r < p.n ? ldg(io.x_in + (size_t)r * p.d + col) : 0.0f;
        }
      } else {
        const int d = p.d, dh = p.Dh;
        if (kNB * nb < 2 * d) {
          const int t = ((kNB * nb) % d % dh) / kNB;
          const int jj = 16 * t + (j & 15);
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int r = 32 * mb + acc_row(i, lane);
            const float2 cs = r < p.n ? ldg((const float2*)p.rope + (size_t)r * (dh / 2) + jj) : make_float2(1.0f, 0.0f);
            pre.a[uu][i] = cs.x;
            pre.b[uu][i] = cs.y;
          }
        }
      }
    }
  }
}

template <int MB, int EPI>
__device__ __forceinline__ void epilogue(KParams& p, const StepIo& io, const float* T, int nb0, int u_lo, int u_hi,
                                         int ub, const EpiPre<EPI>& pre, GemmLds& gl) {
  const int wave = wave_index(), lane = threadIdx.x & 63;
  const int j = lane & 31;
#pragma unroll
  for (int uu = 0; uu < kEpiBatch; ++uu) {
    const int unit = u_lo + wave + kWaves * (ub + uu);
    if (unit >= u_hi) break;
    const int c = unit / MB, mb = unit % MB;
    const int nb = nb0 + c;
    float v[16];
    {
      const float4* src = reinterpret_cast<const float4*>(T + ((size_t)unit * 64 + lane) * 16);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 f = src[q];
        v[4 * q] = f.x;
        v[4 * q + 1] = f.y;
        v[4 * q + 2] = f.z;
        v[4 * q + 3] = f.w;
      }
    }
    if constexpr (EPI != EPI_RESID) {  // the norm's per-row scale
#pragma unroll
      for (int i = 0; i < 16; ++i) v[i] *= gl.rstd[32 * mb + acc_row(i, lane)];
    }
    if constexpr (EPI == EPI_QKV) {
      const int d = p.d, dh = p.Dh;
      const int col = kNB * nb + j;
      if (col < 2 * d) {
        // q or k: this n-block holds dims [16t, 16t+16) (lanes j < 16) and
        // their rotary partners + Dh/2 (lanes j >= 16) of one head.
        const int part = col / d, cq = (kNB * nb) % d, hh = cq / dh, t = (cq % dh) / kNB;
        const int jj = 16 * t + (j & 15);  // pair index < Dh/2
        const int dim = jj + (j < 16 ? 0 : dh / 2);
        bf16* base = part == 0 ? io.q + hh * dh : io.kc + (size_t)hh * p.cap * dh;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = 32 * mb + acc_row(i, lane);
          const float partner = __shfl_xor(v[i], 16, kWave);
          const float cs = pre.a[uu][i], sn = pre.b[uu][i];
          const float outv = j < 16 ? v[i] * cs - partner * sn : v[i] * cs + partner * sn;
          const float nxt = __shfl_down(outv, 1, kWave);
          if (r < p.n && (j & 1) == 0) {
            bf16* dst = part == 0 ? base + (size_t)r * d : base + (size_t)(p.prefix_len + r) * dh;
            st_coherent_bf2(dst + dim, outv, nxt);
          }
        }
      } else {
        const int cv = col - 2 * d, hh = cv / dh, dim = cv % dh;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = 32 * mb + acc_row(i, lane);
          const float nxt = __shfl_down(v[i], 1, kWave);
          if (r < p.n && (j & 1) == 0)
            st_coherent_bf2(io.vc + ((size_t)hh * p.cap + p.prefix_len + r) * dh + dim, v[i], nxt);
        }
      }
    } else if constexpr (EPI == EPI_RESID) {
      const int col = kNB * nb + j;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int r = 32 * mb + acc_row(i, lane);
        const float xn = r < p.n ? pre.a[uu][i] + v[i] : 0.0f;
        if (r < p.n) st_coherent(io.x_out + (size_t)r * p.d + col, xn);
        const float xg = xn * pre.g[uu];
        const float xg1 = __shfl_down(xg, 1, kWave);
        if (r < p.n && (j & 1) == 0) st_coherent_bf2(io.xg_out + (size_t)r * p.d + col, xg, xg1);
        float s = xn * xn;  // sum of squares over the n-block's 32 columns
        s += __shfl_xor(s, 16, kWave);
        s += __shfl_xor(s, 8, kWave);
        s += __shfl_xor(s, 4, kWave);
        s += __shfl_xor(s, 2, kWave);
        s += __shfl_xor(s, 1, kWave);
        if (j == 0 && r < p.n) st_coherent(io.ssq_out + (size_t)nb * p.Mp + r, s);
      }
    } else if constexpr (EPI == EPI_SWIGLU) {
      const int f = 16 * nb + (j & 15);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int r = 32 * mb + acc_row(i, lane);
        const float up = __shfl_xor(v[i], 16, kWave);
        const float hv = v[i] / (1.0f + expf(-v[i])) * up;
        const float nxt = __shfl_down(hv, 1, kWave);
        if (r < p.n && j < 16 && (j & 1) == 0) st_coherent_bf2(io.h + (size_t)r * p.Fp + f, hv, nxt);
      }
    } else {  // EPI_LOGITS
      const int col = kNB * nb + j;
      const bool vcol = col < p.V;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int r = 32 * mb + acc_row(i, lane);
        const bool valid = vcol && r < p.n;
        if (valid && p.logits != nullptr && r >= p.row_lo) stg(p.logits + (size_t)(r - p.row_lo) * p.V + col, v[i]);
        float mv = valid ? v[i] : -INFINITY;
        int mi = valid ? col : 0x7fffffff;
#pragma unroll
        for (int off = 16; off >= 1; off >>= 1) {  // argmax over the n-block's 32 columns
          const float ov = __shfl_xor(mv, off, kWave);
          const int oi = __shfl_xor(mi, off, kWave);
          if (ov > mv || (ov == mv && oi < mi)) {
            mv = ov;
            mi = oi;
          }
        }
        if (j == 0) {
          gl.red_v[r][c] = mv;
          gl.red_i[r][c] = mi;
        }
      }
    }
  }
}

// LM head: per row, the best (value, lowest column) over this workgroup's
// units of the group, into argmax slot `slot` (-inf where it has none).
template <int MB>
__device__ __forceinline__ void logits_units_argmax(KParams& p, int cw, int u_lo, int u_hi, int slot, GemmLds& gl) {
  __syncthreads();
  for (int r = threadIdx.x; r < 32 * MB; r += kThreads) {
    const int mb = r / 32;
    float mv = -INFINITY;
    int mi = 0x7fffffff;
    for (int c = 0; c < cw; ++c) {
      const int u = c * MB + mb;
      if (u < u_lo || u >= u_hi) continue;
      const float v = gl.red_v[r][c];
      const int i = gl.red_i[r][c];
      if (v > mv || (v == mv && i < mi)) {
        mv = v;
        mi = i;
      }
    }
    st_coherent(&p.lm_val[(size_t)slot * p.Mp + r], mv);
    st_coherent(&p.lm_idx[(size_t)slot * p.Mp + r], mi);
  }
}

// After all argmax partials are in: greedy token per node and the accept walk
// (§3.2): node i is reachable when its parent is and its draft token equals
// the target's token after the parent; the result is the deepest reachable
// node (lowest index among equally deep ones).
__device__ __forceinline__ void finish_walk(KParams& p, int entries, GemmLds& gl) {
  const int wave = wave_index(), lane = threadIdx.x & 63;
  for (int r = wave; r < p.n; r += kWaves) {
    float mv = -INFINITY;
    int mi = 0x7fffffff;
    for (int t0 = 0; t0 < entries; t0 += 4 * 64) {
      float v[4];
      int ix[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int t = t0 + 64 * u + lane;
        v[u] = t < entries ? ld_coherent(&p.lm_val[(size_t)t * p.Mp + r]) : -INFINITY;
        ix[u] = t < entries ? ld_coherent(&p.lm_idx[(size_t)t * p.Mp + r]) : 0x7fffffff;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (v[u] > mv || (v[u] == mv && ix[u] < mi)) {
          mv = v[u];
          mi = ix[u];
        }
    }
    wave_argmax(mv, mi);
    if (lane == 0) {
      stg(p.amax + r, mi);
      gl.amax[r] = mi;
    }
  }
  for (int i = threadIdx.x; i < p.n; i += kThreads) {
    gl.tok[i] = ldg(p.tree + i);
    gl.par[i] = ldg(p.tree + 128 + i);
    gl.dep[i] = ldg(p.tree + 256 + i);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const int* tok = gl.tok;
    const int* par = gl.par;
    const int* dep = gl.dep;
    int best = 0, best_depth = 0;
    gl.reach[0] = 1;
    for (int i = 1; i < p.n; ++i) {
      const int pr = par[i];
      const int ok = gl.reach[pr] && (tok[i] == gl.amax[pr]);
      gl.reach[i] = ok;
      if (ok && dep[i] > best_depth) {
        best = i;
        best_depth = dep[i];
      }
    }
    for (int i = best; i >= 0; i = par[i]) gl.reach[dep[i]] = -1 - i;  // path by depth, encoded
    gl.walk_len = best_depth;
    stg(p.accept_len, best_depth);
    stg(p.next_token, gl.amax[best]);
  }
  __syncthreads();
  {
    const int best_depth = gl.walk_len;
    for (int k = threadIdx.x; k < p.n; k += kThreads) {
      const int v = gl.reach[k];
      stg(p.path + k, (k <= best_depth && v < 0) ? -1 - v : -1);
    }
  }
  __syncthreads();
}

// The hand-off of one tile whose sum is in T.  With S > 1 the tile's
// partial goes to memory; when the step has at most one tile per workgroup,
// the S workgroups of the group wait for each other and each adds the S
// partials of its own 1/S of the group's units (in slice order) and runs
// their epilogue; otherwise (no waits inside a phase: a workgroup's later
// tile could be waited for) the group's last workgroup does all of it.  A
// function of its own so that its registers are allocated apart from the
// streaming loops'.  False if a wait ran out.
template <int MB, int EPI>
__device__ __attribute__((noinline, not_tail_called)) bool finish_tile(KParams& pin, int step, int layer, int t,
                                                                      int tr_phase, char* A, GemmLds& gl,
                                                                      int* lds_flag) {
  KParams& p = uniform_params(pin);
  step = wave_uniform(step);
  layer = wave_uniform(layer);
  t = wave_uniform(t);
  tr_phase = wave_uniform(tr_phase);
  const Sync sy = make_sync(p, lds_flag);
  const StepPlan& sp = p.step[step];
  const int S = sp.S, tiles = sp.groups * sp.S;
  const StepIo io = step_io(p, step, layer);
  const int g = t / S, s = t % S;
  const int nb0 = g * sp.cw + (g < sp.n_hi ? g : sp.n_hi);
  const int cw = sp.cw + (g < sp.n_hi ? 1 : 0);
  const int U = cw * MB;
  const int tile_words = U * 1024;
  float* T = reinterpret_cast<float*>(A);
  int u_lo = 0, u_hi = U;
  bool finish = true;
  const bool shared = tiles <= p.G;
  int* cnt = sp.group_cnt + g;
  float* part_g = p.part + (size_t)(nb0 * S) * MB * 1024;
  if (S > 1) {
    float* mine = part_g + (size_t)s * tile_words;
    for (int w = 2 * threadIdx.x; w < tile_words; w += 2 * kThreads) st_coherent2(mine + w, T[w], T[w + 1]);
    if (shared) {
      u_lo = s * U / S;
      u_hi = (s + 1) * U / S;
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      if (threadIdx.x == 0) atomic_add_dev(cnt, 1);
    } else {
      finish = arrive_last(cnt, S, lds_flag);
    }
  }
  EpiPre<EPI> pre;
  if (finish) epilogue_preload<MB, EPI>(p, io, nb0, u_lo, u_hi, 0, pre);
  if constexpr (EPI != EPI_RESID) {
    if (finish) row_scales<MB>(p, io, gl);
  }
  if (S > 1) {
    if (tr_phase >= 0) trace_mark(sy, tr_phase, 6);
    // Group counters are cleared when the pass ends: within a pass a step's
    // counter of a group is used once per layer.
    if (shared && !wait_at_least(sy, cnt, S * (layer + 1))) return false;
    if (finish) {
      // T[units u_lo..u_hi) = sum of the S partials in slice order.  Loads
      // go out in batches of 4 slices x 8 pairs per thread, so the sum costs
      // about S / 4 round trips.
      constexpr int B = 8;
      const int p_lo = u_lo * 512, p_hi = u_hi * 512;  // float2 pairs
      for (int base = p_lo + (int)threadIdx.x; base < p_hi; base += kThreads * B) {
        float2 acc[B];
#pragma unroll
        for (int j = 0; j < B; ++j) acc[j] = make_float2(0.0f, 0.0f);
        for (int s0 = 0; s0 < S; s0 += 4) {
          float2 v[4][B];
#pragma unroll
          for (int k = 0; k < 4; ++k)
#pragma unroll
            for (int j = 0; j < B; ++j) {
              const int idx = base + j * kThreads;
              v[k][j] = (s0 + k < S && idx < p_hi)
                            ? ld_coherent2(part_g + (size_t)(s0 + k) * tile_words + 2 * idx)
                            : make_float2(0.0f, 0.0f);
            }
#pragma unroll
          for (int k = 0; k < 4; ++k)
#pragma unroll
            for (int j = 0; j < B; ++j) {
              acc[j].x += v[k][j].x;
              acc[j].y += v[k][j].y;
            }
        }
#pragma unroll
        for (int j = 0; j < B; ++j) {
          const int idx = base + j * kThreads;
          if (idx < p_hi) {
            T[2 * idx] = acc[j].x;
            T[2 * idx + 1] = acc[j].y;
          }
        }
      }
      __syncthreads();
      if (tr_phase >= 0) trace_mark(sy, tr_phase, 7);
    }
  }
  if (finish) {
    for (int ub = 0; u_lo + wave_index() + kWaves * ub < u_hi; ub += kEpiBatch) {
      if (ub > 0) epilogue_preload<MB, EPI>(p, io, nb0, u_lo, u_hi, ub, pre);
      epilogue<MB, EPI>(p, io, T, nb0, u_lo, u_hi, ub, pre, gl);
    }
    if constexpr (EPI == EPI_LOGITS) {
      const int slot = shared ? t : g;
      logits_units_argmax<MB>(p, cw, u_lo, u_hi, slot, gl);
      if (arrive_last(p.lm_cnt, shared ? tiles : sp.groups, lds_flag)) finish_walk(p, shared ? tiles : sp.groups, gl);
    }
  }
  __syncthreads();
  return true;
}

// One GEMM phase: this workgroup's tiles, each followed by its share of the
// group hand-off and, in the group's last workgroup, the epilogue.
template <int MB, int EPI>
__device__ __attribute__((noinline, not_tail_called)) bool gemm_phase(KParams& pin, int step, int layer,
                                                                     int phase, char* A, GemmLds& gl,
                                                                     int* lds_flag) {
  KParams& p = uniform_params(pin);
  step = wave_uniform(step);
  layer = wave_uniform(layer);
  phase = wave_uniform(phase);
  const Sync sy = make_sync(p, lds_flag);
  const StepPlan& sp = p.step[step];
  const int S = sp.S, tiles = sp.groups * sp.S;
  constexpr int CWM = kMaxCW / MB;
  // The barrier counts arrivals: it is exact only if every workgroup waits
  // at every phase before it arrives again, tile or no tile.
  if ((int)blockIdx.x >= tiles) {
    trace_mark(sy, phase, 0);
    const bool ok = grid_wait(sy, phase, p.G);
    trace_mark(sy, phase, 1);
    return ok;
  }
  bool first = true;
  for (int t = blockIdx.x; t < tiles; t += p.G) {
    const int g = t / S, s = t % S;
    const int nb0 = g * sp.cw + (g < sp.n_hi ? g : sp.n_hi);
    const int cw = sp.cw + (g < sp.n_hi ? 1 : 0);
    const int k0 = (int)((long)s * sp.ksteps / S), k1 = (int)((long)(s + 1) * sp.ksteps / S);
    if (!tile_dispatch<MB, CWM>(cw, p, step, layer, nb0, k0, k1, first ? phase : -1, A, gl, lds_flag))
      return false;
    if (first) trace_mark(sy, phase, 4);
    if (!finish_tile<MB, EPI>(p, step, layer, t, first ? phase : -1, A, gl, lds_flag)) return false;
    first = false;
  }
  trace_mark(sy, phase, 5);
  return true;
}

// ------------------------------------------------------------------ attention

template <int DH>
struct AttnGeom {
  static constexpr int CH = kAttnChunk;  // key positions per LDS tile
  static constexpr int KST = DH + 8;     // K row stride (bf16)
  static constexpr int VST = CH + 8;     // V^T row stride (bf16)
  static constexpr int KS_BYTES = CH * KST * 2;
  static constexpr int VT_BYTES = DH * VST * 2;
  static constexpr int BYTES = KS_BYTES + VT_BYTES;
};

// Stage key positions [p0, p0 + CH) ∩ [lo, hi) of one head into LDS: K
// row-major, V transposed; other rows zero.  Every key comes from the cache:
// the tree's keys and values were written to their slots, already rotated,
// by the QKV phase.
template <int DH>
__device__ __forceinline__ void attn_stage(char* lds, const bf16* kc, const bf16* vc, int p0, int lo,
                                           int hi) {
  using Gm = AttnGeom<DH>;
  bf16* Ks = reinterpret_cast<bf16*>(lds);
  bf16* Vt = reinterpret_cast<bf16*>(lds + Gm::KS_BYTES);
  for (int idx = threadIdx.x; idx < Gm::CH * (DH / 8); idx += kThreads) {
    const int j = idx / (DH / 8), dc = (idx % (DH / 8)) * 8;
    const int pos = p0 + j;
    bf16x8 k0, v0;
    if (pos >= lo && pos < hi) {
      k0 = ldg((const bf16x8*)(kc + (size_t)pos * DH + dc));
      v0 = ldg((const bf16x8*)(vc + (size_t)pos * DH + dc));
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        k0[e] = (bf16)0.0f;
        v0[e] = (bf16)0.0f;
      }
    }
    *(bf16x8*)&Ks[j * Gm::KST + dc] = k0;
#pragma unroll
    for (int e = 0; e < 8; ++e) Vt[(dc + e) * Gm::VST + j] = v0[e];
  }
}

// Tree attention phase: unit (head, split) per workgroup; split s of a head
// covers positions [s T / S, (s + 1) T / S) rounded down to 16, T = prefix_len
// + n.  Node i attends to the prefix and to the cache slots of its
// ancestors-or-self (a 128-bit set per node).  Per unit: S^T = K q^T on the
// matrix cores, online softmax in the log2 domain, O^T += V^T P^T with P split
// into two bf16 halves (P never leaves registers: the S result's lane layout
// is the PV product's k-slot order).  Then the head's splits join and each
// merges its share of the rows.
template <int MB, int DH>
__device__ __attribute__((noinline, not_tail_called)) bool attn_phase(KParams& pin, int layer, int phase, char* lds,
                                                                     int* lds_flag) {
  KParams& p = uniform_params(pin);
  const Sync sy = make_sync(p, lds_flag);
  layer = wave_uniform(layer);
  phase = wave_uniform(phase);
  using Gm = AttnGeom<DH>;
  constexpr int CH = Gm::CH, KSTEPS = DH / 32, DB = DH / 16, KST = Gm::KST, VST = Gm::VST;
  constexpr int RPW = MB > 4 ? 2 : 1;
  const int S = wave_uniform(p.attn_splits);
  const int units = wave_uniform(p.H) * S;
  const int total = wave_uniform(p.prefix_len + p.n);
  const int wave = wave_index(), lane = threadIdx.x & 63, li = lane & 15, g = lane >> 4;
  const int MBr = wave_uniform(p.Mp / 16);
  const size_t kv_layer = (size_t)p.H * p.cap * DH;
  bf16* kcl = p.k_cache + (size_t)layer * kv_layer;
  const bf16* vcl = p.v_cache + (size_t)layer * kv_layer;
  const bf16* qb = p.q + (size_t)layer * p.Mp * p.d;
  bf16* Ks = reinterpret_cast<bf16*>(lds);
  bf16* Vt = reinterpret_cast<bf16*>(lds + Gm::KS_BYTES);

  // The first tile of the first unit is staged before the barrier when it
  // only holds prefix keys (which this pass does not write).
  int u = blockIdx.x;
  bool staged = false;
  if (u < units) {
    const int h = u / S, s = u % S;
    const int lo = (s * total / S) & ~15, hi = s + 1 == S ? total : ((s + 1) * total / S) & ~15;
    const int hi0 = lo + CH < hi ? lo + CH : hi;
    if (lo < hi && hi0 <= p.prefix_len) {
      attn_stage<DH>(lds, kcl + (size_t)h * p.cap * DH, vcl + (size_t)h * p.cap * DH, lo, lo, hi0);
      staged = true;
    }
  }
  trace_mark(sy, phase, 0);
  if (!grid_wait(sy, phase, p.G)) return false;
  trace_mark(sy, phase, 1);

  for (; u < units; u += p.G) {
    const int h = u / S, s = u % S;
    const int lo = (s * total / S) & ~15, hi = s + 1 == S ? total : ((s + 1) * total / S) & ~15;
    bf16* kc = kcl + (size_t)h * p.cap * DH;
    const bf16* vc = vcl + (size_t)h * p.cap * DH;
    // Query fragments (B operand of S^T = K q^T): lane holds row 16 rb + li,
    // dims 32 ks + 8 g + e (queries were rotated by the QKV phase).
    bf16x8 qf[RPW][KSTEPS];
    uint32_t anc[RPW][4];
    float m_run[RPW], l_run[RPW];
    f32x4 oacc[RPW][DB];
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      const int rb = wave + 4 * r;
      const int row = 16 * (rb < MBr ? rb : 0) + li;
      const bf16* qrow = qb + (size_t)row * p.d + h * DH;
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ++ks) qf[r][ks] = ldg((const bf16x8*)(qrow + 32 * ks + 8 * g));
      const uint32_t* ap = (const uint32_t*)(p.tree + 512) + row * 4;
#pragma unroll
      for (int w = 0; w < 4; ++w) anc[r][w] = ldg(ap + w);
      m_run[r] = -INFINITY;
      l_run[r] = 0.0f;
#pragma unroll
      for (int db = 0; db < DB; ++db) oacc[r][db] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    trace_mark(sy, phase, 3);
    for (int p0 = lo; p0 < hi; p0 += CH) {
      const int hi_t = p0 + CH < hi ? p0 + CH : hi;
      if (!staged) {
        __syncthreads();
        attn_stage<DH>(lds, kc, vc, p0, p0, hi_t);
      }
      staged = false;
      __syncthreads();
#pragma unroll
      for (int r = 0; r < RPW; ++r) {
        const int rb = wave + 4 * r;
        if (rb >= MBr) continue;
        for (int c0 = 0; c0 < CH && p0 + c0 < hi_t; c0 += 64) {  // 64 keys per softmax step
          f32x4 sc[4];
#pragma unroll
          for (int jb = 0; jb < 4; ++jb) {
            sc[jb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KSTEPS; ++ks) {
              const bf16x8 a = *(const bf16x8*)&Ks[(c0 + 16 * jb + li) * KST + 32 * ks + 8 * g];
              sc[jb] = mfma16x16x32(a, qf[r][ks], sc[jb]);
            }
          }
          float mx = -INFINITY;
#pragma unroll
          for (int jb = 0; jb < 4; ++jb)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int pos = p0 + c0 + 16 * jb + 4 * g + e;
              const int t = pos - p.prefix_len;
              const bool vis = pos < hi_t && (pos < p.prefix_len ||
                                              (t < p.n && ((anc[r][t >> 5] >> (t & 31)) & 1u)));
              const float sv = vis ? sc[jb][e] * p.scale_log2 : -INFINITY;
              sc[jb][e] = sv;
              mx = fmaxf(mx, sv);
            }
          mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
          mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
          const float m_new = fmaxf(m_run[r], mx);
          const float m_use = (m_new == -INFINITY) ? 0.0f : m_new;
          const float alpha = exp2f(m_run[r] - m_use);
          bf16 ph[4][4], pl[4][4];
          float psum = 0.0f;
#pragma unroll
          for (int jb = 0; jb < 4; ++jb)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float pe = exp2f(sc[jb][e] - m_use);
              ph[jb][e] = f2bf(pe);
              pl[jb][e] = f2bf(pe - bf2f(ph[jb][e]));
              psum += pe;
            }
          psum += __shfl_xor(psum, 16, kWave);
          psum += __shfl_xor(psum, 32, kWave);
          l_run[r] = l_run[r] * alpha + psum;
          m_run[r] = m_new;
#pragma unroll
          for (int db = 0; db < DB; ++db) oacc[r][db] = oacc[r][db] * alpha;
#pragma unroll
          for (int t2 = 0; t2 < 2; ++t2) {
            bf16x8 bph, bpl;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              bph[e] = ph[2 * t2][e];
              bph[4 + e] = ph[2 * t2 + 1][e];
              bpl[e] = pl[2 * t2][e];
              bpl[4 + e] = pl[2 * t2 + 1][e];
            }
#pragma unroll
            for (int db = 0; db < DB; ++db) {
              const bf16* vrow = &Vt[(16 * db + li) * VST + c0 + 32 * t2 + 4 * g];
              const bf16x4 lo4 = *(const bf16x4*)vrow;
              const bf16x4 hi4 = *(const bf16x4*)(vrow + 16);
              bf16x8 av;
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                av[e] = lo4[e];
                av[4 + e] = hi4[e];
              }
              oacc[r][db] = mfma16x16x32(av, bph, oacc[r][db]);
              oacc[r][db] = mfma16x16x32(av, bpl, oacc[r][db]);
            }
          }
        }
      }
    }
    // Per-split results, then join the head's splits and merge this split's
    // share of the rows.
    const size_t head_base = (size_t)h * S * p.Mp;
    const size_t split_base = head_base + (size_t)s * p.Mp;
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      const int rb = wave + 4 * r;
      if (rb >= MBr) continue;
      const int row = 16 * rb + li;
      if (g == 0) st_coherent2(&p.attn_ml[(split_base + row) * 2], m_run[r], l_run[r]);
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        float* dst = &p.attn_o[(split_base + row) * DH + 16 * db + 4 * g];
        st_coherent2(dst, oacc[r][db][0], oacc[r][db][1]);
        st_coherent2(dst + 2, oacc[r][db][2], oacc[r][db][3]);
      }
    }
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) atomic_add_dev(&p.head_cnt[h], 1);
    trace_mark(sy, phase, 4);
    if (!wait_at_least(sy, &p.head_cnt[h], S * (layer + 1))) return false;
    trace_mark(sy, phase, 5);

    const int r_lo = s * p.n / S, r_hi = (s + 1) * p.n / S;
    const int nr = r_hi - r_lo;
    float (*wgt)[kMaxNodes] = reinterpret_cast<float (*)[kMaxNodes]>(lds);
    float (*lsum)[kMaxNodes] = wgt + kAttnMaxSplits;
    for (int idx = threadIdx.x; idx < S * nr; idx += kThreads) {
      const int ss = idx / nr, i = r_lo + idx % nr;
      const float2 ml = ld_coherent2(&p.attn_ml[(head_base + (size_t)ss * p.Mp + i) * 2]);
      wgt[ss][i] = ml.x;
      lsum[ss][i] = ml.y;
    }
    __syncthreads();
    if (threadIdx.x < nr) {
      const int i = r_lo + threadIdx.x;
      float M = -INFINITY;
      for (int ss = 0; ss < S; ++ss) M = fmaxf(M, wgt[ss][i]);
      float L = 0.0f;
      for (int ss = 0; ss < S; ++ss) {
        const float w = exp2f(wgt[ss][i] - M);
        wgt[ss][i] = w;
        L += lsum[ss][i] * w;
      }
      const float inv = 1.0f / L;
      for (int ss = 0; ss < S; ++ss) wgt[ss][i] *= inv;
    }
    __syncthreads();
    bf16* obase = p.o + (size_t)layer * p.Mp * p.d;
    for (int idx = threadIdx.x; idx < nr * (DH / 2); idx += kThreads) {
      const int i = r_lo + idx / (DH / 2), dd = 2 * (idx % (DH / 2));
      float o0 = 0.0f, o1 = 0.0f;
      int ss = 0;
      for (; ss + 4 <= S; ss += 4) {
        float2 v[4];
#pragma unroll
        for (int k = 0; k < 4; ++k)
          v[k] = ld_coherent2(&p.attn_o[(head_base + (size_t)(ss + k) * p.Mp + i) * DH + dd]);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          o0 += v[k].x * wgt[ss + k][i];
          o1 += v[k].y * wgt[ss + k][i];
        }
      }
      for (; ss < S; ++ss) {
        const float2 v = ld_coherent2(&p.attn_o[(head_base + (size_t)ss * p.Mp + i) * DH + dd]);
        o0 += v.x * wgt[ss][i];
        o1 += v.y * wgt[ss][i];
      }
      st_coherent_bf2(obase + (size_t)i * p.d + h * DH + dd, o0, o1);
    }
    __syncthreads();
  }
  return true;
}

// ------------------------------------------------------------------ embed

// Tree preparation (every node's depth, position prefix_len + depth, and
// ancestor-or-self set: its row of the tree masking table) and the residual
// stream's first version: the nodes' embedding rows, with the sums of
// squares of every 32-column n-block.
__device__ __forceinline__ void embed_phase(KParams& p, const TreeArgs& tree, int* par_s) {
  const bf16* E = (const bf16*)(p.packed + p.o_embed);
  if (blockIdx.x == 0) {
    if (threadIdx.x < 128) par_s[threadIdx.x] = threadIdx.x < p.n ? tree.parent[threadIdx.x] : -1;
    __syncthreads();
    if (threadIdx.x < 128) {
      const int i = threadIdx.x;
      int dep = 0;
      uint32_t a[4] = {0u, 0u, 0u, 0u};
      if (i < p.n) {
        for (int j = i; j >= 0; j = par_s[j]) {
          a[j >> 5] |= 1u << (j & 31);
          ++dep;
        }
        --dep;
      }
      st_coherent(&p.tree[i], i < p.n ? tree.tok[i] : 0);
      st_coherent(&p.tree[128 + i], par_s[i]);
      st_coherent(&p.tree[256 + i], dep);
      st_coherent(&p.tree[384 + i], p.prefix_len + dep);
#pragma unroll
      for (int w = 0; w < 4; ++w) st_coherent(&p.tree[512 + i * 4 + w], (int)a[w]);
    }
  }
  const int lane = threadIdx.x & 63;
  for (int m = blockIdx.x; m < p.n; m += p.G) {
    // rotary table row m: (cos, sin) of pos(m) * theta^(-2j/Dh), j < Dh/2
    if (threadIdx.x < p.Dh / 2) {
      int dep = 0;
      for (int j = tree.parent[m]; j >= 0; j = tree.parent[j]) ++dep;
      const int jj = threadIdx.x;
      float sn, cs;
      sincosf((float)(p.prefix_len + dep) * rope_inv_freq(jj, p.Dh, p.log2_theta), &sn, &cs);
      st_coherent2(p.rope + ((size_t)m * (p.Dh / 2) + jj) * 2, cs, sn);
    }
    const bf16* row = E + (size_t)tree.tok[m] * p.d;
    const bf16* g0 = (const bf16*)(p.packed + p.layer0 + p.o_attn_norm);
    for (int c = threadIdx.x; c < p.d; c += kThreads) {
      const float v = bf2f(ldg(row + c));
      st_coherent(&p.x[(size_t)m * p.d + c], v);
      const float xg = v * bf2f(ldg(g0 + c));
      const float xg1 = __shfl_down(xg, 1, kWave);
      if ((c & 1) == 0) st_coherent_bf2(p.xg + (size_t)m * p.d + c, xg, xg1);
      float s = v * v;
      s += __shfl_xor(s, 16, kWave);
      s += __shfl_xor(s, 8, kWave);
      s += __shfl_xor(s, 4, kWave);
      s += __shfl_xor(s, 2, kWave);
      s += __shfl_xor(s, 1, kWave);
      if ((lane & 31) == 0) st_coherent(&p.ssq[(size_t)(c / kNB) * p.Mp + m], s);
    }
  }
}

// ------------------------------------------------------------------ kernel

template <int MB, int DH>
__global__ __launch_bounds__(kThreads, 1) void pass_kernel(const PassParams p_arg, const TreeArgs tree) {
  extern __shared__ __attribute__((aligned(16))) char lds_raw[];
  __shared__ GemmLds gl;
  __shared__ int par_s[128];
  __shared__ int flag;
  // The parameter block is the first kernel argument: read it in place.
  KParams& p = *(KParams*)__builtin_amdgcn_kernarg_segment_ptr();
  if (p.magic != kPassMagic || p.G != p_arg.G || p.n != p_arg.n) {
    if (threadIdx.x == 0 && blockIdx.x == 0) stg(p_arg.status, 3);
    return;  // (uniform over the grid: no workgroup reaches a barrier)
  }
  const Sync sy = make_sync(p, &flag);
  int phase = 0;
  bool ok = true;

  embed_phase(p, tree, par_s);
  grid_arrive(sy, phase);
  ++phase;

  for (int l = 0; l < p.L && ok; ++l) {
    ok = gemm_phase<MB, EPI_QKV>(p, STEP_QKV, l, phase, lds_raw, gl, &flag);
    if (!ok) break;
    grid_arrive(sy, phase++);
    ok = attn_phase<2 * MB, DH>(p, l, phase, lds_raw, &flag);
    if (!ok) break;
    grid_arrive(sy, phase++);
    ok = gemm_phase<MB, EPI_RESID>(p, STEP_O, l, phase, lds_raw, gl, &flag);
    if (!ok) break;
    grid_arrive(sy, phase++);
    ok = gemm_phase<MB, EPI_SWIGLU>(p, STEP_GATE_UP, l, phase, lds_raw, gl, &flag);
    if (!ok) break;
    grid_arrive(sy, phase++);
    ok = gemm_phase<MB, EPI_RESID>(p, STEP_DOWN, l, phase, lds_raw, gl, &flag);
    if (!ok) break;
    grid_arrive(sy, phase++);
  }
  if (ok) {  // final norm + LM head + argmax + accept walk
    if (gemm_phase<MB, EPI_LOGITS>(p, STEP_LM, 0, phase, lds_raw, gl, &flag)) trace_mark(sy, phase, 2);
  }
  // Leave the pass: the last workgroup out resets the barrier and join counters.
  if (arrive_last(p.exit_cnt, p.G, &flag)) {
    if (threadIdx.x < kBarSlots) st_coherent(p.bar + threadIdx.x * kBarStride, 0);
    for (int h = threadIdx.x; h < p.H; h += kThreads) st_coherent(&p.head_cnt[h], 0);
    for (int i = threadIdx.x; i < p.n_group_cnt; i += kThreads) st_coherent(p.group_cnt_all + i, 0);
  }
}

template <int DH>
constexpr size_t dyn_lds_bytes() {
  constexpr size_t attn = AttnGeom<DH>::BYTES;
  constexpr size_t merge = 2 * kAttnMaxSplits * kMaxNodes * 4;
  constexpr size_t a = kAStageBytes;
  constexpr size_t m1 = attn > merge ? attn : merge;
  return m1 > a ? m1 : a;
}

template <int MB, int DH>
hipError_t launch_pass_mb(KParams& p, const TreeArgs& tree, hipStream_t st) {
  static bool attr_set = false;  // per process; the attribute is per function
  const void* fn = (const void*)pass_kernel<MB, DH>;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn_lds_bytes<DH>());
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  void* args[] = {(void*)&p, (void*)&tree};
  return hipLaunchCooperativeKernel(fn, dim3(p.G), dim3(kThreads), args, (unsigned)dyn_lds_bytes<DH>(), st);
}

template <int MB, int DH>
int occupancy_mb() {
  const void* fn = (const void*)pass_kernel<MB, DH>;
  if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn_lds_bytes<DH>()) != hipSuccess)
    return 0;
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, fn, kThreads, dyn_lds_bytes<DH>()) != hipSuccess)
    return 0;
  return blocks;
}

}  // namespace

hipError_t launch_pass(int mb32, KParams& p, const TreeArgs& tree, hipStream_t st) {
#define LLMCAD_PASS_CASE(M)                                                 \
  case M:                                                                   \
    return p.Dh == 128 ? launch_pass_mb<M, 128>(p, tree, st)                \
                       : launch_pass_mb<M, 64>(p, tree, st);
  switch (mb32) {
    LLMCAD_PASS_CASE(1)
    LLMCAD_PASS_CASE(2)
    LLMCAD_PASS_CASE(4)
    default:
      return hipErrorInvalidValue;
  }
#undef LLMCAD_PASS_CASE
}

int pass_occupancy(int mb32, int dh) {
#define LLMCAD_OCC_CASE(M) \
  case M:                  \
    return dh == 128 ? occupancy_mb<M, 128>() : occupancy_mb<M, 64>();
  switch (mb32) {
    LLMCAD_OCC_CASE(1)
    LLMCAD_OCC_CASE(2)
    LLMCAD_OCC_CASE(4)
    default:
      return 0;
  }
#undef LLMCAD_OCC_CASE
}

size_t pass_lds_bytes(int mb32, int dh) {
  (void)mb32;
  return dh == 128 ? dyn_lds_bytes<128>() : dyn_lds_bytes<64>();
}

}  // namespace llmcad
