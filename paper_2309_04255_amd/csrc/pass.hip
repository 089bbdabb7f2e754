// The whole verification pass (§3.2 of arXiv 2309.04255) as one persistent
// launch.
//
// Why one launch: a pass is a chain of five dependent steps per layer, each
// streaming tens to hundreds of MB of weights.  As separate kernels every
// step pays a ramp-up and a drain; here every workgroup (one per CU, all
// resident: cooperative launch) walks the phases in order and meets the
// others at a grid barrier between phases.  Weights never depend on the
// previous phase, so each workgroup issues the first weight loads of its next
// phase before waiting at the barrier, and HBM keeps streaming meanwhile.
//
// Phases: embed + tree prep; per layer QKV projection (RMSNorm prologue) ->
// tree attention (rotary embedding at each node's position, ancestor mask) ->
// O projection (+residual) -> gate/up (RMSNorm prologue, SwiGLU epilogue) ->
// down projection (+residual); then final RMSNorm + LM head + argmax, and the
// accept walk in the workgroup that completes the argmax.
//
// GEMM phases: the output columns are 16-wide n-blocks (one MFMA each).
// Workgroup g owns c = N_blocks / G whole n-blocks over the full K, so its
// epilogue needs nothing from other workgroups; the remaining R = N_blocks mod
// G n-blocks are shared stream-K style (every workgroup gets an equal run of
// their k-steps), finished by the last contributor, which adds the partials
// in k order (bit-reproducible).  Runs over the remainder come first so their
// hand-off latency overlaps the main block's streaming.  Inside a workgroup
// the four waves take interleaved k-steps and their partial sums are added in
// LDS in a fixed order.
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

// How a GEMM phase forms its A operand, and what its epilogue does.
enum Prologue { PRO_BF16 = 0, PRO_NORM = 1 };  // bf16 activations | RMSNorm of fp32 x
enum Epilogue { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_LOGITS = 3 };
constexpr int kTraceWgs = 8;  // workgroups that record phase timestamps

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

// ------------------------------------------------------------------ sync

struct Sync {
  int* bar;
  int* status;
  int limit;
  int* lds_flag;
  long long* trace;  // [phase][6] timestamps of this workgroup, or null
};

__device__ __forceinline__ Sync make_sync(KParams& p, int* lds_flag) {
  Sync s;
  s.bar = p.bar;
  s.status = p.status;
  s.limit = p.spin_limit;
  s.lds_flag = lds_flag;
  s.trace = p.trace != nullptr && (int)blockIdx.x < kTraceWgs
                ? p.trace + (size_t)blockIdx.x * (2 + 5 * p.L) * 6
                : nullptr;
  return s;
}

// Diagnostics: wall-clock (100 MHz) marks per phase: 0 = barrier wait
// entered, 1 = wait over, 2 = phase work done; GEMM phases also mark 3 =
// operand prologue done, 4 = weight streaming of the last segment done,
// 5 = last epilogue done.
__device__ __forceinline__ void trace_mark(const Sync& s, int phase, int k) {
  if (s.trace != nullptr && threadIdx.x == 0) stg(s.trace + phase * 6 + k, (long long)wall_clock64());
}

// End of a phase: this workgroup's stores have completed, then one
// device-scope increment on its barrier counter (workgroup g counts on
// counter g % kBarSlots, so arrivals do not serialise on one address).
__device__ __forceinline__ void grid_arrive(const Sync& s, int phase) {
  trace_mark(s, phase, 2);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0)
    atomic_add_dev(s.bar + (blockIdx.x % kBarSlots) * kBarStride, 1);
}

// Waits until all G workgroups have arrived `phase` times; one wave polls all
// counters.  False (to all threads) if the bounded spin ran out.
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

struct GemmDesc {
  const bf16x8* w;   // packed matrix, n-block major
  int nbt, ks;       // n-blocks, k-steps per n-block
  const bf16* a;     // PRO_BF16: [Mp][lda]
  int lda;
  const float* x;    // PRO_NORM: [Mp][d]
  const float* ssq;  // PRO_NORM: [d/16][Mp]
  const bf16* gain;  // PRO_NORM: [d]
};

struct EpiArgs {
  bf16* q;            // EPI_QKV: [Mp][d] queries after the rotary embedding
  bf16* kc;           // EPI_QKV: K cache of this layer [H][cap][Dh]
  bf16* vc;           // EPI_QKV: V cache of this layer [H][cap][Dh]
  const float* x_in;  // EPI_RESID: [Mp][d]
  float* x_out;       // EPI_RESID: [Mp][d]
  float* ssq_out;     // EPI_RESID: [d/16][Mp]
  bf16* h;            // EPI_SWIGLU: [Mp][Fp]
  float* logits;      // EPI_LOGITS: rows [row_lo, n), or null
  int row_lo;
};

template <int MB, int PRO>
struct AStage;
template <int MB>
struct AStage<MB, PRO_BF16> {
  bf16x8 a[MB];
};
template <int MB>
struct AStage<MB, PRO_NORM> {
  float4 x[MB][2];
  bf16x8 g;
};

// Register pipeline depth: ~192 VGPRs of stages, 2..16 k-steps.
template <int MB, int PRO, int C>
constexpr int pipe_depth() {
  constexpr int per = 4 * C + (PRO == PRO_BF16 ? 4 * MB : 8 * MB + 4);
  constexpr int d = 192 / per;
  return d < 2 ? 2 : (d > 16 ? 16 : d);
}

template <int MB, int PRO, int C>
struct Pipe {
  static constexpr int D = pipe_depth<MB, PRO, C>();
  bf16x8 bw[D][C];
  AStage<MB, PRO> as[D];
  const bf16x8* wt;  // first n-block's blocks + lane
  int ks;            // blocks between consecutive n-blocks
  int s0, ns;        // this wave's first k-step and number of k-steps
};

template <int MB, int PRO, int C>
__device__ __forceinline__ void pipe_setup(Pipe<MB, PRO, C>& P, const GemmDesc& g, int nb0, int k0,
                                           int k1) {
  const int wave = wave_index(), lane = threadIdx.x & 63;
  P.wt = g.w + (size_t)nb0 * g.ks * 64 + lane;
  P.ks = g.ks;
  P.s0 = wave_uniform(k0 + wave);
  P.ns = wave_uniform(P.s0 < k1 ? (k1 - P.s0 + kWaves - 1) / kWaves : 0);
}

template <int MB, int PRO, int C>
__device__ __forceinline__ void pipe_load_b(Pipe<MB, PRO, C>& P, int slot, int i) {
  const int s = P.s0 + kWaves * i;
#pragma unroll
  for (int c = 0; c < C; ++c) P.bw[slot][c] = ldg(P.wt + ((size_t)c * P.ks + s) * 64);
}

template <int MB, int PRO, int C>
__device__ __forceinline__ void pipe_load_a(Pipe<MB, PRO, C>& P, const GemmDesc& g, int d, int slot,
                                            int i) {
  const int lane = threadIdx.x & 63, lrow = lane & 15, kg = lane >> 4;
  const int k = kStepK * (P.s0 + kWaves * i) + 8 * kg;
  if constexpr (PRO == PRO_BF16) {
#pragma unroll
    for (int rb = 0; rb < MB; ++rb)
      P.as[slot].a[rb] = ldg((const bf16x8*)(g.a + (size_t)(16 * rb + lrow) * g.lda + k));
  } else {
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) {
      const float* xr = g.x + (size_t)(16 * rb + lrow) * d + k;
      P.as[slot].x[rb][0] = ldg((const float4*)xr);
      P.as[slot].x[rb][1] = ldg((const float4*)(xr + 4));
    }
    P.as[slot].g = ldg((const bf16x8*)(g.gain + k));
  }
}

template <int MB, int PRO, int C>
__device__ __forceinline__ void pipe_compute(Pipe<MB, PRO, C>& P, int slot, f32x4 (&acc)[MB][C],
                                             const float (&rstd)[MB]) {
#pragma unroll
  for (int rb = 0; rb < MB; ++rb) {
    bf16x8 a;
    if constexpr (PRO == PRO_BF16) {
      a = P.as[slot].a[rb];
    } else {
      const float xs[8] = {P.as[slot].x[rb][0].x, P.as[slot].x[rb][0].y, P.as[slot].x[rb][0].z,
                           P.as[slot].x[rb][0].w, P.as[slot].x[rb][1].x, P.as[slot].x[rb][1].y,
                           P.as[slot].x[rb][1].z, P.as[slot].x[rb][1].w};
#pragma unroll
      for (int e = 0; e < 8; ++e) a[e] = f2bf(xs[e] * rstd[rb] * bf2f(P.as[slot].g[e]));
    }
#pragma unroll
    for (int c = 0; c < C; ++c) acc[rb][c] = mfma16x16x32(a, P.bw[slot][c], acc[rb][c]);
  }
}

// Runs the wave's k-steps as a software pipeline of D register stages.
// Every stage is loaded (weights, then the A operand) D steps ahead of its
// use, and loads are issued unconditionally (clamped to the last step) so
// the number in flight is the same on every path.  The scheduling fences keep
// each stage's compute after the previous stage's reload: the compiler's
// wait before a compute then only covers that stage's own loads, and the
// (D - 1) younger stages stay in flight.
// `hook` runs (in every wave) once the first stages are in flight; the first
// pipeline of a phase computes the RMSNorm scales there, so their loads
// overlap the weight stream.
template <int MB, int PRO, int C, class Hook>
__device__ __forceinline__ void pipe_run(Pipe<MB, PRO, C>& P, const GemmDesc& g, int d,
                                         f32x4 (&acc)[MB][C], const float (&rstd)[MB], Hook&& hook) {
  constexpr int D = Pipe<MB, PRO, C>::D;
#pragma unroll
  for (int rb = 0; rb < MB; ++rb)
#pragma unroll
    for (int c = 0; c < C; ++c) acc[rb][c] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int ns = P.ns;  // wave-uniform
  if (ns > 0) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      const int st = u < ns ? u : ns - 1;
      pipe_load_b(P, u, st);
      pipe_load_a(P, g, d, u, st);
      __builtin_amdgcn_sched_barrier(0);  // stages issue in order
    }
  }
  hook();
  __builtin_amdgcn_sched_barrier(0);
  if (ns == 0) return;
  for (int i = 0; i < ns; i += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      __builtin_amdgcn_sched_barrier(0);
      if (i + u < ns) pipe_compute(P, u, acc, rstd);
      __builtin_amdgcn_sched_barrier(0);
      const int nx = i + u + D < ns ? i + u + D : ns - 1;
      pipe_load_b(P, u, nx);
      pipe_load_a(P, g, d, u, nx);
    }
  }
  __builtin_amdgcn_sched_barrier(0);
}

// Sum the waves' partial tiles into tileS [16 MB][16 C (+4)] in wave order.
template <int MB, int C>
__device__ __forceinline__ void reduce_waves(float* tileS, const f32x4 (&acc)[MB][C]) {
  constexpr int TS = 16 * C + 4;
  const int wave = wave_index(), lane = threadIdx.x & 63, lrow = lane & 15, kg = lane >> 4;
  for (int w = 0; w < kWaves; ++w) {
    if (wave == w) {
#pragma unroll
      for (int rb = 0; rb < MB; ++rb)
#pragma unroll
        for (int c = 0; c < C; ++c)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float* dst = &tileS[(16 * rb + 4 * kg + i) * TS + 16 * c + lrow];
            *dst = (w == 0) ? acc[rb][c][i] : *dst + acc[rb][c][i];
          }
    }
    __syncthreads();
  }
}

// Workgroup whose stream-K run contains flat k-step position q.
__device__ __forceinline__ int owner_of(long q, long W, int G) {
  return (int)(((q + 1) * G + W - 1) / W) - 1;
}

struct GemmLds {
  float part_ss[256];         // rstd prologue: [256 / ROWS][ROWS]
  float red_v[kMaxNodes][8];  // argmax per (row, n-block)
  int red_i[kMaxNodes][8];
  int reach[kMaxNodes];
  int amax[kMaxNodes];
  int tok[kMaxNodes];  // accept walk: the tree, staged from the workspace
  int par[kMaxNodes];
  int dep[kMaxNodes];
  int walk_len;
  float best_v[kMaxNodes];  // LM head: the workgroup's best column per row
  int best_i[kMaxNodes];
};

// Rotary embedding frequency of dim pair (j, j + Dh/2): theta^(-2j/Dh).
__device__ __forceinline__ float rope_inv_freq(int j, int Dh, float log2_theta) {
  return exp2f(-(2.0f * (float)j / (float)Dh) * log2_theta);
}

// Epilogue of C n-blocks [nb0, nb0 + C) held in tileS: writes the phase's
// outputs with device-coherent stores.  lm_entry: argmax partial slot.
template <int MB, int EPI, int C>
__device__ __forceinline__ void epilogue(KParams& p, const EpiArgs& e, float* tileS, int nb0,
                                         int lm_entry, GemmLds& gl) {
  constexpr int ROWS = 16 * MB, COLS = 16 * C, TS = COLS + 4;
  const int lane = threadIdx.x & 63;
  if constexpr (EPI == EPI_QKV) {
    // One thread per (row, column pair cc, cc + 8) of an n-block.  q and k
    // n-blocks hold rotary pairs 8 columns apart (PACK_QKV_ROPE): rotate at
    // the node's position, then store q, and k into the node's cache slot.
    // v n-blocks are plain.  Stores go out in adjacent pairs of dims (this
    // lane and the next).
    const int d = p.d, dh = p.Dh, half = dh / 2;
    for (int idx = threadIdx.x; idx < ROWS * (COLS / 2); idx += kThreads) {
      const int r = idx / (COLS / 2), ps = idx % (COLS / 2);
      const int cc = kNB * (ps / 8) + (ps % 8);
      const int col = kNB * nb0 + cc;
      const float a = tileS[r * TS + cc], b = tileS[r * TS + cc + 8];
      const bool store = r < p.n && (ps & 1) == 0;
      if (col < 2 * d) {
        const int part = col / d, cq = col % d, hh = cq / dh, w = cq % dh;
        const int j = 8 * (w / kNB) + (w % kNB);  // < Dh/2
        const int pos = r < p.n ? ldg(p.tree + 384 + r) : 0;
        float sn, cs;
        sincosf((float)pos * rope_inv_freq(j, dh, p.log2_theta), &sn, &cs);
        const float lo = a * cs - b * sn, hi = b * cs + a * sn;
        const float lo1 = __shfl_down(lo, 1, kWave), hi1 = __shfl_down(hi, 1, kWave);
        if (store) {
          bf16* dst = part == 0 ? e.q + (size_t)r * d + hh * dh
                                : e.kc + ((size_t)hh * p.cap + p.prefix_len + r) * dh;
          st_coherent_bf2(dst + j, lo, lo1);
          st_coherent_bf2(dst + j + half, hi, hi1);
        }
      } else {
        const int j = col - 2 * d, hh = j / dh, dd = j % dh;
        const float a1 = __shfl_down(a, 1, kWave), b1 = __shfl_down(b, 1, kWave);
        if (store) {
          bf16* dst = e.vc + ((size_t)hh * p.cap + p.prefix_len + r) * dh + dd;
          st_coherent_bf2(dst, a, a1);
          st_coherent_bf2(dst + 8, b, b1);
        }
      }
    }
  } else if constexpr (EPI == EPI_RESID) {
    for (int idx = threadIdx.x; idx < ROWS * COLS; idx += kThreads) {
      const int r = idx / COLS, cc = idx % COLS;
      const int col = kNB * nb0 + cc;
      float xn = 0.0f;
      if (r < p.n) {
        xn = ldg(e.x_in + (size_t)r * p.d + col) + tileS[r * TS + cc];
        st_coherent(&e.x_out[(size_t)r * p.d + col], xn);
      }
      // sum of squares over the 16 columns of this n-block (16 consecutive lanes)
      float s = xn * xn;
      s += __shfl_xor(s, 8, kWave);
      s += __shfl_xor(s, 4, kWave);
      s += __shfl_xor(s, 2, kWave);
      s += __shfl_xor(s, 1, kWave);
      if ((lane & 15) == 0) st_coherent(&e.ssq_out[(size_t)(nb0 + cc / kNB) * p.Mp + r], s);
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    for (int idx = threadIdx.x; idx < ROWS * C * 8; idx += kThreads) {
      const int r = idx / (C * 8), rem = idx % (C * 8), i = rem / 8, j = rem % 8;
      const float gt = tileS[r * TS + kNB * i + j], up = tileS[r * TS + kNB * i + 8 + j];
      const float hv = gt / (1.0f + expf(-gt)) * up;
      const float nxt = __shfl_down(hv, 1, kWave);
      if (r < p.n && (j & 1) == 0) st_coherent_bf2(e.h + (size_t)r * p.Fp + 8 * (nb0 + i) + j, hv, nxt);
    }
  } else {  // EPI_LOGITS
    for (int idx = threadIdx.x; idx < ROWS * COLS; idx += kThreads) {
      const int r = idx / COLS, cc = idx % COLS;
      const int col = kNB * nb0 + cc;
      const bool valid = r < p.n && col < p.V;
      const float v = tileS[r * TS + cc];
      if (valid && e.logits != nullptr && r >= e.row_lo) stg(e.logits + (size_t)(r - e.row_lo) * p.V + col, v);
      float mv = valid ? v : -INFINITY;
      int mi = valid ? col : 0x7fffffff;
#pragma unroll
      for (int off = 8; off >= 1; off >>= 1) {  // argmax over the n-block's 16 columns
        const float ov = __shfl_xor(mv, off, kWave);
        const int oi = __shfl_xor(mi, off, kWave);
        if (ov > mv || (ov == mv && oi < mi)) {
          mv = ov;
          mi = oi;
        }
      }
      if ((lane & 15) == 0) {
        gl.red_v[r][cc / kNB] = mv;
        gl.red_i[r][cc / kNB] = mi;
      }
    }
    __syncthreads();
    for (int r = threadIdx.x; r < ROWS; r += kThreads) {
      float mv = -INFINITY;
      int mi = 0x7fffffff;
      for (int c = 0; c < C; ++c) {
        const float v = gl.red_v[r][c];
        const int i = gl.red_i[r][c];
        if (v > mv || (v == mv && i < mi)) {
          mv = v;
          mi = i;
        }
      }
      if (lm_entry >= 0) {  // a remainder n-block: its own argmax entry
        st_coherent(&p.lm_val[(size_t)lm_entry * p.Mp + r], mv);
        st_coherent(&p.lm_idx[(size_t)lm_entry * p.Mp + r], mi);
      } else if (lm_entry == -2 || mv > gl.best_v[r] || (mv == gl.best_v[r] && mi < gl.best_i[r])) {
        gl.best_v[r] = mv;  // main block: best over its sub-blocks (-2: first sub-block)
        gl.best_i[r] = mi;
      }
    }
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

// Warms L2 with the first 16 KiB of weights each wave will read: blocks of
// n-blocks [nb0, nb0 + nbs) at the wave's k-steps k0 + wave, + 4, ... (< k1),
// in the order the pipeline consumes them, so that HBM keeps streaming while
// the workgroup waits at a barrier.  The loaded values are folded into a
// token after the wait (prefetch_fold) so the loads stay live.
struct Prefetch {
  bf16x8 v[16];
};
__device__ __forceinline__ void l2_prefetch(Prefetch& pf, const bf16x8* w, int ks, int nb0, int nbs,
                                            int k0, int k1) {
  const int wave = wave_index(), lane = threadIdx.x & 63;
  const int s0 = k0 + wave;
  const int ns = s0 < k1 ? (k1 - s0 + kWaves - 1) / kWaves : 0;
  const int total = ns * nbs;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int it = i < total ? i : (total > 0 ? total - 1 : 0);
    const int c = it % nbs, s = s0 + kWaves * (it / nbs);
    const size_t blk = total > 0 ? ((size_t)(nb0 + c) * ks + s) : 0;
    pf.v[i] = ldg(w + blk * 64 + lane);
  }
}
__device__ __forceinline__ uint32_t prefetch_fold(const Prefetch& pf) {
  uint32_t tok = 0;
#pragma unroll
  for (int i = 0; i < 16; ++i) tok ^= __builtin_bit_cast(uint32_t, (__bf16 __attribute__((ext_vector_type(2)))){pf.v[i][0], pf.v[i][1]});
  return tok;
}


// The GEMM steps of the pass and their operands.
enum Step { STEP_QKV = 0, STEP_O = 1, STEP_GATE_UP = 2, STEP_DOWN = 3, STEP_LM = 4 };

__device__ __forceinline__ void step_operands(KParams& p, int step, int l, GemmDesc& g, EpiArgs& e) {
  const size_t xsz = (size_t)p.Mp * p.d, ssz = (size_t)p.d_nb * p.Mp;
  const char* lw = p.packed + p.layer0 + (long long)l * p.layer_bytes;
  g = GemmDesc{};
  e = EpiArgs{};
  switch (step) {
    case STEP_QKV:  // RMSNorm(x_2l) -> q, k (raw) and v (to the cache)
      g.w = (const bf16x8*)(lw + p.o_qkv);
      g.nbt = p.qkv_nb;
      g.ks = p.ks_d;
      g.x = p.x + (size_t)(2 * l) * xsz;
      g.ssq = p.ssq + (size_t)(2 * l) * ssz;
      g.gain = (const bf16*)(lw + p.o_attn_norm);
      e.q = p.q + (size_t)l * p.Mp * p.d;
      e.kc = p.k_cache + (size_t)l * p.H * p.cap * p.Dh;
      e.vc = p.v_cache + (size_t)l * p.H * p.cap * p.Dh;
      break;
    case STEP_O:  // x_2l+1 = x_2l + o W_o^T
      g.w = (const bf16x8*)(lw + p.o_o);
      g.nbt = p.d_nb;
      g.ks = p.ks_d;
      g.a = p.o + (size_t)l * p.Mp * p.d;
      g.lda = p.d;
      e.x_in = p.x + (size_t)(2 * l) * xsz;
      e.x_out = p.x + (size_t)(2 * l + 1) * xsz;
      e.ssq_out = p.ssq + (size_t)(2 * l + 1) * ssz;
      break;
    case STEP_GATE_UP:  // h = SwiGLU(RMSNorm(x_2l+1))
      g.w = (const bf16x8*)(lw + p.o_gu);
      g.nbt = p.gu_nb;
      g.ks = p.ks_d;
      g.x = p.x + (size_t)(2 * l + 1) * xsz;
      g.ssq = p.ssq + (size_t)(2 * l + 1) * ssz;
      g.gain = (const bf16*)(lw + p.o_ffn_norm);
      e.h = p.h + (size_t)l * p.Mp * p.Fp;
      break;
    case STEP_DOWN:  // x_2l+2 = x_2l+1 + h W_down^T
      g.w = (const bf16x8*)(lw + p.o_down);
      g.nbt = p.d_nb;
      g.ks = p.ks_f;
      g.a = p.h + (size_t)l * p.Mp * p.Fp;
      g.lda = p.Fp;
      e.x_in = p.x + (size_t)(2 * l + 1) * xsz;
      e.x_out = p.x + (size_t)(2 * l + 2) * xsz;
      e.ssq_out = p.ssq + (size_t)(2 * l + 2) * ssz;
      break;
    default:  // STEP_LM: logits = RMSNorm(x_2L) W_lm^T
      g.w = (const bf16x8*)(p.packed + p.o_lm);
      g.nbt = p.v_nb;
      g.ks = p.ks_d;
      g.x = p.x + (size_t)(2 * p.L) * xsz;
      g.ssq = p.ssq + (size_t)(2 * p.L) * ssz;
      g.gain = (const bf16*)(p.packed + p.o_final_norm);
      e.logits = p.logits;
      e.row_lo = p.row_lo;
      break;
  }
}

// RMSNorm scales of the rows (this lane's row 16 rb + lane % 16 for each row
// block rb): 1 / sqrt(mean of squares + eps), from the per-n-block sums of
// squares the producing phase wrote.
template <int MB>
__device__ __forceinline__ void row_scales(KParams& p, const GemmDesc& g, GemmLds& gl, float (&rstd)[MB]) {
  constexpr int ROWS = 16 * MB, CHK = 256 / ROWS;
  const int lrow = threadIdx.x & 15;
  const int dn = p.d_nb;
  if (threadIdx.x < CHK * ROWS) {
    const int r = threadIdx.x % ROWS, ch = threadIdx.x / ROWS;
    const int t0 = ch * dn / CHK, t1 = (ch + 1) * dn / CHK;
    float ss = 0.0f;
    int t = t0;
    for (; t + 4 <= t1; t += 4) {
      const float v0 = ldg(g.ssq + (size_t)t * p.Mp + r), v1 = ldg(g.ssq + (size_t)(t + 1) * p.Mp + r);
      const float v2 = ldg(g.ssq + (size_t)(t + 2) * p.Mp + r), v3 = ldg(g.ssq + (size_t)(t + 3) * p.Mp + r);
      ss += v0;
      ss += v1;
      ss += v2;
      ss += v3;
    }
    for (; t < t1; ++t) ss += ldg(g.ssq + (size_t)t * p.Mp + r);
    gl.part_ss[ch * ROWS + r] = ss;
  }
  __syncthreads();
#pragma unroll
  for (int rb = 0; rb < MB; ++rb) {
    const int row = 16 * rb + lrow;
    float ss = 0.0f;
#pragma unroll
    for (int ch = 0; ch < CHK; ++ch) ss += gl.part_ss[ch * ROWS + row];
    rstd[rb] = 1.0f / sqrtf(ss * p.inv_d + p.eps);
  }
  __syncthreads();
}

template <int MB>
struct RowScale {
  float v[MB];
};

// Widest main-block sub-block (n-blocks streamed together, sharing one pass
// over the A operand) that the registers allow at MB row blocks.
template <int MB>
constexpr int max_width() {
  return MB <= 2 ? 8 : (MB <= 4 ? 4 : 2);
}

// CM whole n-blocks [nb0, nb0 + CM) over the full K.  A function of its own
// per width, so each width gets its own register allocation.  When need_rs
// is set the RMSNorm scales are computed here, once the first weight stages
// are in flight; the scales used are returned.
template <int MB, int PRO, int EPI, int CM>
__device__ __attribute__((noinline, not_tail_called)) RowScale<MB> main_block(
    KParams& pin, int step, int layer, int nb0, RowScale<MB> rs, int need_rs, float* tileS, GemmLds& gl,
    int lm_entry) {
  KParams& p = uniform_params(pin);
  GemmDesc g;
  EpiArgs e;
  step_operands(p, wave_uniform(step), wave_uniform(layer), g, e);
  nb0 = wave_uniform(nb0);
  lm_entry = wave_uniform(lm_entry);
  bool need = wave_uniform(need_rs) != 0;
  float rstd[MB];
#pragma unroll
  for (int rb = 0; rb < MB; ++rb) rstd[rb] = rs.v[rb];
  auto hook = [&]() {
    if constexpr (PRO == PRO_NORM) {
      if (need) row_scales<MB>(p, g, gl, rstd);
    }
  };
  Pipe<MB, PRO, CM> P;
  pipe_setup(P, g, nb0, 0, g.ks);
  f32x4 acc[MB][CM];
  pipe_run(P, g, p.d, acc, rstd, hook);
  reduce_waves<MB, CM>(tileS, acc);
  epilogue<MB, EPI, CM>(p, e, tileS, nb0, lm_entry, gl);
  __syncthreads();
  RowScale<MB> out;
#pragma unroll
  for (int rb = 0; rb < MB; ++rb) out.v[rb] = rstd[rb];
  return out;
}

template <int MB, int PRO, int EPI, int W>
__device__ __forceinline__ RowScale<MB> main_dispatch(int w, KParams& p, int step, int layer, int nb0,
                                                      RowScale<MB> rs, int need_rs, float* tileS,
                                                      GemmLds& gl, int lm) {
  if constexpr (W >= 1) {
    if (w == W) return main_block<MB, PRO, EPI, W>(p, step, layer, nb0, rs, need_rs, tileS, gl, lm);
    return main_dispatch<MB, PRO, EPI, W - 1>(w, p, step, layer, nb0, rs, need_rs, tileS, gl, lm);
  } else {
    return rs;
  }
}

// One GEMM phase: warm L2 with the first weights, wait at the barrier, then
// the remainder runs (stream-K, one n-block per segment) and the main block
// (whole n-blocks over the full K, in sub-blocks of 4, 3, 2 or 1 n-blocks).
template <int MB, int PRO, int EPI>
__device__ __attribute__((noinline, not_tail_called)) bool gemm_phase(KParams& pin, int step, int layer, int phase,
                                                     float* tileS, GemmLds& gl, int* lds_flag) {
  KParams& p = uniform_params(pin);
  const Sync sy = make_sync(p, lds_flag);
  GemmDesc g;
  EpiArgs e;
  step_operands(p, wave_uniform(step), wave_uniform(layer), g, e);
  phase = wave_uniform(phase);
  constexpr int ROWS = 16 * MB;
  const int G = p.G, gi = blockIdx.x;
  const int c = g.nbt / G, R = g.nbt - c * G;
  const long Wr = (long)R * g.ks;
  const long rbeg = (long)gi * Wr / G, rend = (long)(gi + 1) * Wr / G;

  {
    Prefetch pf;
    if (rbeg < rend) {
      const int t = (int)(rbeg / g.ks), k0 = (int)(rbeg % g.ks);
      const int k1 = (int)(k0 + (rend - rbeg) < g.ks ? k0 + (rend - rbeg) : g.ks);
      l2_prefetch(pf, g.w, g.ks, c * G + t, 1, k0, k1);
    } else if (c > 0) {
      l2_prefetch(pf, g.w, g.ks, gi * c, c < max_width<MB>() ? c : max_width<MB>(), 0, g.ks);
    } else {
      l2_prefetch(pf, g.w, g.ks, 0, 1, 0, 0);
    }
    trace_mark(sy, phase, 0);
    if (!grid_wait(sy, phase, G)) return false;
    trace_mark(sy, phase, 1);
    const uint32_t tok = prefetch_fold(pf);
    if (tok == 0x9e3779b9u && p.G < 0) stg(p.status + 1, (int)tok);  // keeps the prefetch loads
  }

  float rstd[MB];
#pragma unroll
  for (int rb = 0; rb < MB; ++rb) rstd[rb] = 1.0f;
  // RMSNorm scales: computed by the first pipeline of the phase once its
  // first stages are in flight.
  bool need_rstd = PRO == PRO_NORM;
  auto rstd_hook = [&]() {
    if constexpr (PRO == PRO_NORM) {
      if (!need_rstd) return;
      need_rstd = false;
      row_scales<MB>(p, g, gl, rstd);
    }
  };

  // Remainder n-blocks (stream-K), one n-block per segment.
  for (long pos = rbeg; pos < rend;) {
    const int t = (int)(pos / g.ks), k0 = (int)(pos % g.ks);
    const int k1 = (int)(k0 + (rend - pos) < g.ks ? k0 + (rend - pos) : g.ks);
    const int nb = c * G + t;
    {
      Pipe<MB, PRO, 1> P1;
      pipe_setup(P1, g, nb, k0, k1);
      f32x4 acc[MB][1];
      pipe_run(P1, g, p.d, acc, rstd, rstd_hook);
      reduce_waves<MB, 1>(tileS, acc);
    }
    constexpr int TS = 16 + 4;
    bool finish = true;
    if (!(k0 == 0 && k1 == g.ks)) {
      const int slot = (pos == rbeg) ? 0 : 1;
      float* mine = p.part + ((size_t)gi * 2 + slot) * ROWS * kNB;
      for (int idx = 2 * threadIdx.x; idx < ROWS * kNB; idx += 2 * kThreads)
        st_coherent2(mine + idx, tileS[(idx / kNB) * TS + idx % kNB], tileS[(idx / kNB) * TS + idx % kNB + 1]);
      const long tile_lo = (long)t * g.ks, tile_hi = tile_lo + g.ks - 1;
      const int g_lo = owner_of(tile_lo, Wr, G), g_hi = owner_of(tile_hi, Wr, G);
      int contributors = 0;
      for (int gg = g_lo; gg <= g_hi; ++gg)
        contributors += ((long)gg * Wr / G < (long)(gg + 1) * Wr / G) ? 1 : 0;
      finish = arrive_last(&p.tile_cnt[nb], contributors, sy.lds_flag);
      if (finish) {
        for (int idx = 2 * threadIdx.x; idx < ROWS * kNB; idx += 2 * kThreads) {
          float s0 = 0.0f, s1 = 0.0f;
          for (int gg = g_lo; gg <= g_hi; ++gg) {
            const long gb = (long)gg * Wr / G;
            if (gb == (long)(gg + 1) * Wr / G) continue;  // empty run
            const int sl = (gg == g_lo && gb < tile_lo) ? 1 : 0;
            const float2 v = ld_coherent2(p.part + ((size_t)gg * 2 + sl) * ROWS * kNB + idx);
            s0 += v.x;
            s1 += v.y;
          }
          tileS[(idx / kNB) * TS + idx % kNB] = s0;
          tileS[(idx / kNB) * TS + idx % kNB + 1] = s1;
        }
        __syncthreads();
      }
    }
    if (finish) {
      epilogue<MB, EPI, 1>(p, e, tileS, nb, G + t, gl);
      if constexpr (EPI == EPI_LOGITS) {
        if (arrive_last(p.lm_cnt, G + R, sy.lds_flag)) finish_walk(p, G + R, gl);
      }
    }
    __syncthreads();
    pos += k1 - k0;
  }

  // Main block: n-blocks [gi c, (gi + 1) c) over the full K.  For the LM head
  // the workgroup's argmax entry is the best over its sub-blocks.
  trace_mark(sy, phase, 3);
  for (int done = 0; done < c;) {
    const int w = c - done < max_width<MB>() ? c - done : max_width<MB>();
    const int nb0 = gi * c + done;
    const int lm = done == 0 ? -2 : -1;
    RowScale<MB> rs;
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) rs.v[rb] = rstd[rb];
    rs = main_dispatch<MB, PRO, EPI, max_width<MB>()>(w, p, step, layer, nb0, rs, need_rstd ? 1 : 0,
                                                       tileS, gl, lm);
    need_rstd = false;
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) rstd[rb] = rs.v[rb];
    done += w;
  }
  trace_mark(sy, phase, 4);
  if constexpr (EPI == EPI_LOGITS) {
    for (int r = threadIdx.x; r < ROWS; r += kThreads) {
      const size_t at = (size_t)gi * p.Mp + r;
      st_coherent(&p.lm_val[at], c > 0 ? gl.best_v[r] : -INFINITY);
      st_coherent(&p.lm_idx[at], c > 0 ? gl.best_i[r] : 0x7fffffff);
    }
    if (arrive_last(p.lm_cnt, G + R, sy.lds_flag)) finish_walk(p, G + R, gl);
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
    if (threadIdx.x == 0)
      atomic_add_dev(&p.head_cnt[h], 1);
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
// stream's first version: the nodes' embedding rows.
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
  for (int m = blockIdx.x; m < p.Mp; m += p.G) {
    const bool valid = m < p.n;
    const bf16* row = E + (size_t)(valid ? tree.tok[m] : 0) * p.d;
    for (int c = threadIdx.x; c < p.d; c += kThreads) {
      const float v = valid ? bf2f(ldg(row + c)) : 0.0f;
      st_coherent(&p.x[(size_t)m * p.d + c], v);
      float s = v * v;
      s += __shfl_xor(s, 8, kWave);
      s += __shfl_xor(s, 4, kWave);
      s += __shfl_xor(s, 2, kWave);
      s += __shfl_xor(s, 1, kWave);
      if ((lane & 15) == 0) st_coherent(&p.ssq[(size_t)(c / kNB) * p.Mp + m], s);
    }
  }
}

// ------------------------------------------------------------------ kernel

template <int MB, int DH>
constexpr int pass_lds_bytes() {
  constexpr int attn = AttnGeom<DH>::BYTES;
  constexpr int merge = 2 * kAttnMaxSplits * kMaxNodes * 4;
  constexpr int tile = 16 * MB * (16 * max_width<MB>() + 4) * 4;
  constexpr int m1 = attn > merge ? attn : merge;
  return m1 > tile ? m1 : tile;
}

template <int MB, int DH>
__global__ __launch_bounds__(kThreads, 1) void pass_kernel(const PassParams p_arg, const TreeArgs tree) {
  __shared__ __attribute__((aligned(16))) char lds_raw[pass_lds_bytes<MB, DH>()];
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
  float* tileS = reinterpret_cast<float*>(lds_raw);
  int phase = 0;
  bool ok = true;

  embed_phase(p, tree, par_s);
  grid_arrive(sy, phase);
  ++phase;

  for (int l = 0; l < p.L && ok; ++l) {
    ok = gemm_phase<MB, PRO_NORM, EPI_QKV>(p, STEP_QKV, l, phase, tileS, gl, &flag);
    if (!ok) break;
    grid_arrive(sy, phase++);
    ok = attn_phase<MB, DH>(p, l, phase, lds_raw, &flag);
    if (!ok) break;
    grid_arrive(sy, phase++);
    ok = gemm_phase<MB, PRO_BF16, EPI_RESID>(p, STEP_O, l, phase, tileS, gl, &flag);
    if (!ok) break;
    grid_arrive(sy, phase++);
    ok = gemm_phase<MB, PRO_NORM, EPI_SWIGLU>(p, STEP_GATE_UP, l, phase, tileS, gl, &flag);
    if (!ok) break;
    grid_arrive(sy, phase++);
    ok = gemm_phase<MB, PRO_BF16, EPI_RESID>(p, STEP_DOWN, l, phase, tileS, gl, &flag);
    if (!ok) break;
    grid_arrive(sy, phase++);
  }
  if (ok) {  // final norm + LM head + argmax + accept walk
    if (gemm_phase<MB, PRO_NORM, EPI_LOGITS>(p, STEP_LM, 0, phase, tileS, gl, &flag))
      trace_mark(sy, phase, 2);
  }
  // Leave the pass: the last workgroup out resets the barrier and join counters.
  if (arrive_last(p.exit_cnt, p.G, &flag)) {
    if (threadIdx.x < kBarSlots) st_coherent(p.bar + threadIdx.x * kBarStride, 0);
    for (int h = threadIdx.x; h < p.H; h += kThreads) st_coherent(&p.head_cnt[h], 0);
  }
}

template <int MB, int DH>
hipError_t launch_pass_mb(KParams& p, const TreeArgs& tree, hipStream_t st) {
  void* args[] = {(void*)&p, (void*)&tree};
  return hipLaunchCooperativeKernel((const void*)pass_kernel<MB, DH>, dim3(p.G), dim3(kThreads), args,
                                    0, st);
}

template <int MB, int DH>
int occupancy_mb() {
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, (const void*)pass_kernel<MB, DH>, kThreads,
                                                   0) != hipSuccess)
    return 0;
  return blocks;
}

}  // namespace

hipError_t launch_pass(int mb, KParams& p, const TreeArgs& tree, hipStream_t st) {
#define LLMCAD_PASS_CASE(M)                                                 \
  case M:                                                                   \
    return p.Dh == 128 ? launch_pass_mb<M, 128>(p, tree, st)                \
                       : launch_pass_mb<M, 64>(p, tree, st);
  switch (mb) {
    LLMCAD_PASS_CASE(1)
    LLMCAD_PASS_CASE(2)
    LLMCAD_PASS_CASE(3)
    LLMCAD_PASS_CASE(4)
    LLMCAD_PASS_CASE(8)
    default:
      return hipErrorInvalidValue;
  }
#undef LLMCAD_PASS_CASE
}

int pass_occupancy(int mb, int dh) {
#define LLMCAD_OCC_CASE(M) \
  case M:                  \
    return dh == 128 ? occupancy_mb<M, 128>() : occupancy_mb<M, 64>();
  switch (mb) {
    LLMCAD_OCC_CASE(1)
    LLMCAD_OCC_CASE(2)
    LLMCAD_OCC_CASE(3)
    LLMCAD_OCC_CASE(4)
    LLMCAD_OCC_CASE(8)
    default:
      return 0;
  }
#undef LLMCAD_OCC_CASE
}

}  // namespace llmcad
