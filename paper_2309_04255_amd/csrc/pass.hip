// The whole verification pass (§3.2 of arXiv 2309.04255) as one persistent
// launch.
//
// Why one launch: a pass is a chain of ~5 dependent steps per layer, each
// streaming tens to hundreds of MB of weights.  As separate kernels every step
// pays a ramp-up and a drain; here every workgroup (one per CU, all resident:
// cooperative launch) walks the phases in order and meets the others at a
// grid barrier between phases.  Weights never depend on the previous phase,
// so each workgroup issues the first weight loads of its next phase *before*
// waiting at the barrier, and HBM keeps streaming while the barrier settles.
//
// Phases: embed + tree prep; per layer QKV (+RMSNorm, rotary, KV write) ->
// tree attention -> O (+residual) -> gate/up (+RMSNorm, SwiGLU) -> down
// (+residual); then final RMSNorm + LM head + argmax, and the accept walk in
// the last tile to finish.
//
// GEMM phases are stream-K: the (64-column tile, 32-wide k-step) grid of a
// matrix is cut into G equal contiguous runs, one per workgroup, so every
// workgroup streams the same number of weight bytes.  A tile covered by
// several runs is finished by the last contributor, which adds the partials
// in k order (bit-reproducible).
//
// Coherence without cache maintenance: every buffer handed from one phase to
// the next is written once per pass at its own address with device-coherent
// stores and read after the barrier with ordinary (cacheable) loads, so no L2
// can hold an older copy; buffers reused within a pass (partials) are read
// with device-coherent loads.  Barriers and per-head joins are monotonic
// counters polled with bounded spins: a wait that exceeds its bound records
// an error status and the workgroup leaves the pass, so no wave can hang.
#include <math.h>

#include "device.h"
#include "kernels.h"
#include "layout.h"

namespace llmcad {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kTraceWgs = 8;  // workgroups that record phase timestamps

__device__ __forceinline__ void st_coherent_bf2(bf16* p, float a, float b) {  // p 4-byte aligned
  const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, f2bf(a));
  const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, f2bf(b));
  __hip_atomic_store((uint32_t*)p, lo | (hi << 16), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ------------------------------------------------------------------ barrier

struct Sync {
  int* bar;
  int* status;
  int limit;
  int* lds_flag;
  long long* trace;  // [phase][3] timestamps of this workgroup, or null
};

// Diagnostics: wall-clock (100 MHz) marks per phase: 0 = barrier wait entered,
// 1 = wait over, 2 = phase work done; GEMM phases also mark 3 = operand
// prologue done, 4 = weight streaming of the last segment done, 5 = last
// epilogue done.
__device__ __forceinline__ void trace_mark(const Sync& s, int phase, int k) {
  if (s.trace != nullptr && threadIdx.x == 0) s.trace[phase * 6 + k] = (long long)wall_clock64();
}

// The grid barrier is spread over kBarSlots counters (one per 128-byte line)
// so that arrivals do not serialise on one address: workgroup g counts on
// slot g % kBarSlots, and a waiter polls all slots with one wave.
constexpr int kBarSlots = 16;
constexpr int kBarStride = 32;  // ints between slots

// Arrival at the end of a phase: this workgroup's stores are complete, then
// one device-scope increment.
__device__ __forceinline__ void grid_arrive(const Sync& s, int phase) {
  trace_mark(s, phase, 2);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0)
    __hip_atomic_fetch_add(s.bar + (blockIdx.x % kBarSlots) * kBarStride, 1, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

// Waits until every barrier slot has seen `phase` arrivals from each of its
// workgroups; false (to all threads) if the bounded spin ran out.
__device__ __forceinline__ bool grid_wait(const Sync& s, int phase, int G) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    const int slots = G < kBarSlots ? G : kBarSlots;
    const int per = G / kBarSlots + (lane < G % kBarSlots ? 1 : 0);
    const int want = lane < slots ? phase * (G < kBarSlots ? 1 : per) : 0;
    int* slot = s.bar + (lane < slots ? lane : 0) * kBarStride;
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

// Waits until *c >= target; false (to all threads) if the bounded spin ran out.
__device__ __forceinline__ bool wait_at_least(const Sync& s, int* c, int target) {
  if (threadIdx.x == 0) {
    int ok = 1, spins = 0;
    while (ld_coherent(c) < target) {
      __builtin_amdgcn_s_sleep(2);
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
  const bf16x8* w;  // packed matrix
  int tiles, ks;    // 64-column tiles, 32-wide k-steps per tile
  // A operand
  const bf16* a;    // PRO_BF16: [Mp][lda]
  int lda;
  const float* x;   // PRO_NORM: [Mp][d]
  const float* ssq; // PRO_NORM: [d/64][Mp]
  const bf16* gain; // PRO_NORM: [d]
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

template <int MB, int PRO, int D>
struct Pipe {
  bf16x8 bw[D][4];
  AStage<MB, PRO> as[D];
  const bf16x8* wt;  // tile base + lane
  int s0, ns;        // this wave's first k-step, number of k-steps
};

template <int MB, int PRO, int D>
__device__ __forceinline__ void pipe_setup(Pipe<MB, PRO, D>& P, const GemmDesc& g, int tile, int k0,
                                           int k1) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  P.wt = g.w + (size_t)tile * g.ks * 256 + lane;
  P.s0 = k0 + wave;
  P.ns = P.s0 < k1 ? (k1 - P.s0 + kWaves - 1) / kWaves : 0;
}

template <int MB, int PRO, int D>
__device__ __forceinline__ void pipe_load_b(Pipe<MB, PRO, D>& P, int slot, int i) {
  const int s = P.s0 + kWaves * i;
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) P.bw[slot][nb] = P.wt[(size_t)s * 256 + nb * 64];
}

template <int MB, int PRO, int D>
__device__ __forceinline__ void pipe_load_a(Pipe<MB, PRO, D>& P, const GemmDesc& g, int d, int slot,
                                            int i) {
  const int lane = threadIdx.x & 63, lrow = lane & 15, kg = lane >> 4;
  const int k = 32 * (P.s0 + kWaves * i) + 8 * kg;
  if constexpr (PRO == PRO_BF16) {
#pragma unroll
    for (int rb = 0; rb < MB; ++rb)
      P.as[slot].a[rb] = *(const bf16x8*)(g.a + (size_t)(16 * rb + lrow) * g.lda + k);
  } else {
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) {
      const float* xr = g.x + (size_t)(16 * rb + lrow) * d + k;
      P.as[slot].x[rb][0] = *(const float4*)xr;
      P.as[slot].x[rb][1] = *(const float4*)(xr + 4);
    }
    P.as[slot].g = *(const bf16x8*)(g.gain + k);
  }
}

template <int MB, int PRO, int D>
__device__ __forceinline__ void pipe_compute(Pipe<MB, PRO, D>& P, int slot, f32x4 (&acc)[MB][4],
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
    for (int nb = 0; nb < 4; ++nb) acc[rb][nb] = mfma16x16x32(a, P.bw[slot][nb], acc[rb][nb]);
  }
}

// Runs the wave's k-steps.  If b_ready, the first D weight stages were issued
// before (across a barrier).  Loads are issued unconditionally (clamped to the
// last step) so the number in flight is the same on every path.
template <int MB, int PRO, int D>
__device__ __forceinline__ void pipe_run(Pipe<MB, PRO, D>& P, const GemmDesc& g, int d, bool b_ready,
                                         f32x4 (&acc)[MB][4], const float (&rstd)[MB]) {
#pragma unroll
  for (int rb = 0; rb < MB; ++rb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[rb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (P.ns == 0) return;
  if (!b_ready) {
#pragma unroll
    for (int u = 0; u < D; ++u) pipe_load_b(P, u, u < P.ns ? u : P.ns - 1);
  }
#pragma unroll
  for (int u = 0; u < D; ++u) pipe_load_a(P, g, d, u, u < P.ns ? u : P.ns - 1);
  for (int i = 0; i < P.ns; i += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      if (i + u < P.ns) pipe_compute(P, u, acc, rstd);
      const int nx = i + u + D < P.ns ? i + u + D : P.ns - 1;
      pipe_load_b(P, u, nx);
      pipe_load_a(P, g, d, u, nx);
    }
  }
}

// Sum the waves' partial tiles into tileS (fixed wave order).
template <int MB>
__device__ __forceinline__ void reduce_waves(float (*tileS)[68], const f32x4 (&acc)[MB][4]) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, lrow = lane & 15, kg = lane >> 4;
  for (int w = 0; w < kWaves; ++w) {
    if (wave == w) {
#pragma unroll
      for (int rb = 0; rb < MB; ++rb)
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float* dst = &tileS[16 * rb + 4 * kg + i][16 * nb + lrow];
            *dst = (w == 0) ? acc[rb][nb][i] : *dst + acc[rb][nb][i];
          }
    }
    __syncthreads();
  }
}

// Workgroup whose stream-K run contains flat k-step position q.
__device__ __forceinline__ int owner_of(long q, long W, int G) {
  return (int)(((q + 1) * G + W - 1) / W) - 1;
}

// ------------------------------------------------------------------ epilogues

struct EpiQkv {
  bf16* q;        // [Mp][d]
  bf16* kc;       // [H][cap][Dh] of this layer
  bf16* vc;
  const int* pos; // [n]
};
struct EpiResid {
  const float* x_in;  // [Mp][d]
  float* x_out;       // [Mp][d]
  float* ssq_out;     // [d/64][Mp]
};
struct EpiSwiglu {
  bf16* h;  // [Mp][Fp]
};
struct EpiLogits {
  float* logits;
  int row_lo;
};

}  // namespace

namespace {

template <int MB>
struct PassLds {
  float tileS[MB * 16][68];
  float part_ss[256 / (MB * 16) > 0 ? 256 / (MB * 16) : 1][MB * 16];
  int reach[kMaxNodes];
  int amax[kMaxNodes];
};

// One GEMM phase.  Issues this workgroup's first weight loads, then waits for
// `target` arrivals at the grid barrier, then runs its stream-K run.
template <int MB, int PRO, int EPI, int D>
__device__ __forceinline__ bool gemm_phase(const PassParams& p, const GemmDesc& g, const Sync& sy,
                                           int target, PassLds<MB>& lds, int layer, const void* epi) {
  constexpr int ROWS = MB * 16;
  const int G = p.G;
  const long W = (long)g.tiles * g.ks;
  const long begin = (long)blockIdx.x * W / G, end = (long)(blockIdx.x + 1) * W / G;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, lrow = lane & 15;

  Pipe<MB, PRO, D> P;
  long pos = begin;
  if (pos < end) {
    const int t = (int)(pos / g.ks), k0 = (int)(pos % g.ks);
    const int k1 = (int)((long)k0 + (end - pos) < g.ks ? k0 + (end - pos) : g.ks);
    pipe_setup(P, g, t, k0, k1);
    if (P.ns > 0) {
#pragma unroll
      for (int u = 0; u < D; ++u) pipe_load_b(P, u, u < P.ns ? u : P.ns - 1);
    }
  }
  trace_mark(sy, target / p.G, 0);
  if (!grid_wait(sy, target / p.G, p.G)) return false;
  trace_mark(sy, target / p.G, 1);

  float rstd[MB];
#pragma unroll
  for (int rb = 0; rb < MB; ++rb) rstd[rb] = 1.0f;
  if constexpr (PRO == PRO_NORM) {
    constexpr int CH = 256 / ROWS;
    const int dt = p.d_tiles;
    if (threadIdx.x < CH * ROWS) {
      const int r = threadIdx.x % ROWS, c = threadIdx.x / ROWS;
      const int t0 = c * dt / CH, t1 = (c + 1) * dt / CH;
      float ss = 0.0f;
      int t = t0;
      for (; t + 4 <= t1; t += 4) {
        const float v0 = g.ssq[(size_t)t * p.Mp + r], v1 = g.ssq[(size_t)(t + 1) * p.Mp + r];
        const float v2 = g.ssq[(size_t)(t + 2) * p.Mp + r], v3 = g.ssq[(size_t)(t + 3) * p.Mp + r];
        ss += v0;
        ss += v1;
        ss += v2;
        ss += v3;
      }
      for (; t < t1; ++t) ss += g.ssq[(size_t)t * p.Mp + r];
      lds.part_ss[c][r] = ss;
    }
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) {
      const int row = 16 * rb + lrow;
      float ss = 0.0f;
#pragma unroll
      for (int c = 0; c < CH; ++c) ss += lds.part_ss[c][row];
      rstd[rb] = 1.0f / sqrtf(ss * p.inv_d + p.eps);
    }
  }

  const int ph = target / G;
  trace_mark(sy, ph, 3);
  bool first = true;
  while (pos < end) {
    const int t = (int)(pos / g.ks), k0 = (int)(pos % g.ks);
    const int k1 = (int)((long)k0 + (end - pos) < g.ks ? k0 + (end - pos) : g.ks);
    if (!first) pipe_setup(P, g, t, k0, k1);
    f32x4 acc[MB][4];
    pipe_run(P, g, p.d, first, acc, rstd);
    trace_mark(sy, ph, 4);
    reduce_waves<MB>(lds.tileS, acc);
    bool finish = true;
    if (!(k0 == 0 && k1 == g.ks)) {
      // Partial tile: store it, count the arrival, the last contributor sums.
      const int slot = (pos == begin) ? 0 : 1;
      float* mine = p.part + ((size_t)blockIdx.x * 2 + slot) * ROWS * 64;
      for (int idx = 2 * threadIdx.x; idx < ROWS * 64; idx += 512)
        st_coherent2(mine + idx, lds.tileS[idx >> 6][idx & 63], lds.tileS[idx >> 6][(idx & 63) + 1]);
      const long tile_lo = (long)t * g.ks, tile_hi = tile_lo + g.ks - 1;
      const int g_lo = owner_of(tile_lo, W, G), g_hi = owner_of(tile_hi, W, G);
      int contributors = 0;  // workgroups with a non-empty run inside the tile
      for (int gg = g_lo; gg <= g_hi; ++gg)
        contributors += ((long)gg * W / G < (long)(gg + 1) * W / G) ? 1 : 0;
      finish = arrive_last(&p.tile_cnt[t], contributors, sy.lds_flag);
      if (finish) {
        for (int idx = 2 * threadIdx.x; idx < ROWS * 64; idx += 512) {
          float s0 = 0.0f, s1 = 0.0f;
          for (int gg = g_lo; gg <= g_hi; ++gg) {
            const long gb = (long)gg * W / G;
            if (gb == (long)(gg + 1) * W / G) continue;  // empty run
            const int sl = (gg == g_lo && gb < tile_lo) ? 1 : 0;
            const float2 v = ld_coherent2(p.part + ((size_t)gg * 2 + sl) * ROWS * 64 + idx);
            s0 += v.x;
            s1 += v.y;
          }
          lds.tileS[idx >> 6][idx & 63] = s0;
          lds.tileS[idx >> 6][(idx & 63) + 1] = s1;
        }
        __syncthreads();
      }
    }
    if (finish) {
      if constexpr (EPI == EPI_QKV) {
        const EpiQkv& e = *(const EpiQkv*)epi;
        const int tiles_per_head = p.Dh / 64;
        const int per_part = p.H * tiles_per_head;
        const int part = t / per_part, rr = t % per_part;
        const int hh = rr / tiles_per_head, b = rr % tiles_per_head;
        const int half = p.Dh / 2;
        const int jj = 32 * b + (lane & 31);
        const int j = lane < 32 ? jj : half + jj;
        const float inv_freq = exp2f(-(2.0f * (float)jj / (float)p.Dh) * p.log2_theta);
        for (int r = wave; r < p.n; r += kWaves) {
          const float v = lds.tileS[r][lane];
          float out = v;
          if (part < 2) {
            const float partner = lds.tileS[r][lane ^ 32];
            float sn, cs;
            sincosf((float)e.pos[r] * inv_freq, &sn, &cs);
            out = lane < 32 ? v * cs - partner * sn : v * cs + partner * sn;
          }
          const float nxt = __shfl_down(out, 1, kWave);
          if ((lane & 1) == 0) {
            bf16* dst;
            if (part == 0)
              dst = e.q + (size_t)r * p.d + hh * p.Dh + j;
            else
              dst = (part == 1 ? e.kc : e.vc) + ((size_t)hh * p.cap + p.prefix_len + r) * p.Dh + j;
            st_coherent_bf2(dst, out, nxt);
          }
        }
      } else if constexpr (EPI == EPI_RESID) {
        const EpiResid& e = *(const EpiResid*)epi;
        const int col = 64 * t + lane;
        for (int r = wave; r < ROWS; r += kWaves) {
          float xn = 0.0f;
          if (r < p.n) {
            xn = e.x_in[(size_t)r * p.d + col] + lds.tileS[r][lane];
            st_coherent(&e.x_out[(size_t)r * p.d + col], xn);
          }
          const float s = wave_sum(xn * xn);
          if (lane == 0) st_coherent(&e.ssq_out[(size_t)t * p.Mp + r], s);
        }
      } else if constexpr (EPI == EPI_SWIGLU) {
        const EpiSwiglu& e = *(const EpiSwiglu*)epi;
        const int c = lane & 31;
        for (int r = wave; r < p.n; r += kWaves) {
          const float gt = lds.tileS[r][c], up = lds.tileS[r][32 + c];
          const float hv = gt / (1.0f + expf(-gt)) * up;
          const float nxt = __shfl_down(hv, 1, kWave);
          if (lane < 32 && (lane & 1) == 0) st_coherent_bf2(e.h + (size_t)r * p.Fp + 32 * t + c, hv, nxt);
        }
      } else {  // EPI_LOGITS
        const EpiLogits& e = *(const EpiLogits*)epi;
        const int col = 64 * t + lane;
        for (int r = wave; r < ROWS; r += kWaves) {
          const bool valid = r < p.n && col < p.V;
          const float v = lds.tileS[r][lane];
          if (valid && e.logits != nullptr && r >= e.row_lo) e.logits[(size_t)(r - e.row_lo) * p.V + col] = v;
          float mv = valid ? v : -INFINITY;
          int mi = valid ? col : 0x7fffffff;
          wave_argmax(mv, mi);
          if (lane == 0) {
            st_coherent(&p.lm_val[(size_t)t * p.Mp + r], mv);
            st_coherent(&p.lm_idx[(size_t)t * p.Mp + r], mi);
          }
        }
        if (arrive_last(p.lm_cnt, g.tiles, sy.lds_flag)) {
          for (int r = wave; r < p.n; r += kWaves) {
            float mv = -INFINITY;
            int mi = 0x7fffffff;
            for (int t0 = 0; t0 < g.tiles; t0 += 4 * 64) {
              float v[4];
              int ix[4];
#pragma unroll
              for (int u = 0; u < 4; ++u) {
                const int tt = t0 + 64 * u + lane;
                v[u] = tt < g.tiles ? ld_coherent(&p.lm_val[(size_t)tt * p.Mp + r]) : -INFINITY;
                ix[u] = tt < g.tiles ? ld_coherent(&p.lm_idx[(size_t)tt * p.Mp + r]) : 0x7fffffff;
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
              p.amax[r] = mi;
              lds.amax[r] = mi;
            }
          }
          __syncthreads();
          if (threadIdx.x == 0) {
            const int* tok = p.tree;
            const int* par = p.tree + 128;
            const int* dep = p.tree + 256;
            int best = 0, best_depth = 0;
            lds.reach[0] = 1;
            for (int i = 1; i < p.n; ++i) {
              const int pr = par[i];
              const int ok = lds.reach[pr] && (tok[i] == lds.amax[pr]);
              lds.reach[i] = ok;
              if (ok && dep[i] > best_depth) {
                best = i;
                best_depth = dep[i];
              }
            }
            for (int k = 0; k < p.n; ++k) p.path[k] = -1;
            for (int i = best; i >= 0; i = par[i]) p.path[dep[i]] = i;
            *p.accept_len = best_depth;
            *p.next_token = lds.amax[best];
          }
        }
      }
      __syncthreads();
    }
    trace_mark(sy, ph, 5);
    pos += k1 - k0;
    first = false;
  }
  (void)layer;
  return true;
}

// ------------------------------------------------------------------ attention

template <int MB, int DH>
struct AttnLds {
  static constexpr int CH = kAttnChunk;
  static constexpr int KST = DH + 8;
  static constexpr int VST = CH + 8;
  static constexpr int KS_BYTES = CH * KST * 2, VT_BYTES = DH * VST * 2;
  static constexpr int MERGE_BYTES = 2 * kAttnMaxSplits * kMaxNodes * 4;
  static constexpr int BYTES = KS_BYTES + VT_BYTES > MERGE_BYTES ? KS_BYTES + VT_BYTES : MERGE_BYTES;
};

// Stage key positions [p0, p0 + 64) of head h into LDS (K row-major, V
// transposed); positions outside [lo, hi) are zero.
template <int DH>
__device__ __forceinline__ void attn_stage(char* lds, const bf16* kc, const bf16* vc, int p0, int lo,
                                           int hi) {
  constexpr int CH = kAttnChunk, KST = DH + 8, VST = CH + 8;
  bf16* Ks = reinterpret_cast<bf16*>(lds);
  bf16* Vt = reinterpret_cast<bf16*>(lds + CH * KST * 2);
  for (int idx = threadIdx.x; idx < CH * DH / 8; idx += kThreads) {
    const int j = idx / (DH / 8), dc = (idx % (DH / 8)) * 8;
    const int pos = p0 + j;
    bf16x8 kv, vv;
    if (pos >= lo && pos < hi) {
      kv = *(const bf16x8*)(kc + (size_t)pos * DH + dc);
      vv = *(const bf16x8*)(vc + (size_t)pos * DH + dc);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        kv[e] = (bf16)0.0f;
        vv[e] = (bf16)0.0f;
      }
    }
    *(bf16x8*)&Ks[j * KST + dc] = kv;
#pragma unroll
    for (int e = 0; e < 8; ++e) Vt[(dc + e) * VST + j] = vv[e];
  }
}

// Tree attention phase: unit (head, split) per workgroup; positions of a split
// are [s * T / S, (s + 1) * T / S) rounded to 16, T = prefix_len + n.
template <int MB, int DH>
__device__ __forceinline__ bool attn_phase(const PassParams& p, int layer, const Sync& sy, int target,
                                           char* lds) {
  constexpr int CH = kAttnChunk, KSTEPS = DH / 32, DB = DH / 16, KST = DH + 8, VST = CH + 8;
  constexpr int RPW = MB > 4 ? 2 : 1;
  const int S = p.attn_splits;
  const int units = p.H * S;
  const int total = p.prefix_len + p.n;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, li = lane & 15, g = lane >> 4;
  const int d = p.H * DH;
  const size_t kv_layer = (size_t)p.H * p.cap * DH;
  const bf16* kcl = p.k_cache + (size_t)layer * kv_layer;
  const bf16* vcl = p.v_cache + (size_t)layer * kv_layer;
  bf16* Ks = reinterpret_cast<bf16*>(lds);
  bf16* Vt = reinterpret_cast<bf16*>(lds + CH * KST * 2);

  // Units of this workgroup: blockIdx.x, blockIdx.x + G, ...  The first
  // chunk of the first unit is staged before the barrier when it only holds
  // prefix positions (which this pass does not write).
  int u = blockIdx.x;
  bool staged = false;
  if (u < units) {
    const int h = u / S, s = u % S;
    const int lo = (s * total / S) & ~15, hi = s + 1 == S ? total : ((s + 1) * total / S) & ~15;
    if (lo < hi && hi <= p.prefix_len) {
      attn_stage<DH>(lds, kcl + (size_t)h * p.cap * DH, vcl + (size_t)h * p.cap * DH, lo, lo, hi);
      staged = true;
    }
  }
  trace_mark(sy, target / p.G, 0);
  if (!grid_wait(sy, target / p.G, p.G)) return false;
  trace_mark(sy, target / p.G, 1);

  const bf16* qbase = p.q + (size_t)layer * p.Mp * d;
  for (; u < units; u += p.G) {
    const int h = u / S, s = u % S;
    const int lo = (s * total / S) & ~15, hi = s + 1 == S ? total : ((s + 1) * total / S) & ~15;
    const bf16* kc = kcl + (size_t)h * p.cap * DH;
    const bf16* vc = vcl + (size_t)h * p.cap * DH;
    bf16x8 qf[RPW][KSTEPS];
    uint32_t anc[RPW][4];
    float m_run[RPW], l_run[RPW];
    f32x4 oacc[RPW][DB];
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      const int rb = wave + 4 * r;
      const int row = 16 * (rb < MB ? rb : 0) + li;
      const bf16* qr = qbase + (size_t)row * d + h * DH;
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ++ks) qf[r][ks] = *(const bf16x8*)(qr + 32 * ks + 8 * g);
      const uint32_t* ap = (const uint32_t*)(p.tree + 512) + row * 4;
#pragma unroll
      for (int w = 0; w < 4; ++w) anc[r][w] = ap[w];
      m_run[r] = -INFINITY;
      l_run[r] = 0.0f;
#pragma unroll
      for (int db = 0; db < DB; ++db) oacc[r][db] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    for (int p0 = lo; p0 < hi; p0 += CH) {
      if (!staged) {
        __syncthreads();
        attn_stage<DH>(lds, kc, vc, p0, lo, hi);
      }
      staged = false;
      __syncthreads();
#pragma unroll
      for (int r = 0; r < RPW; ++r) {
        const int rb = wave + 4 * r;
        if (rb >= MB) continue;
        f32x4 sc[4];
#pragma unroll
        for (int jb = 0; jb < 4; ++jb) {
          sc[jb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks < KSTEPS; ++ks) {
            const bf16x8 a = *(const bf16x8*)&Ks[(16 * jb + li) * KST + 32 * ks + 8 * g];
            sc[jb] = mfma16x16x32(a, qf[r][ks], sc[jb]);
          }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int jb = 0; jb < 4; ++jb)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int pos = p0 + 16 * jb + 4 * g + e;
            const int t = pos - p.prefix_len;
            const bool vis = pos < hi && (pos < p.prefix_len ||
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
            const bf16* vrow = &Vt[(16 * db + li) * VST + 32 * t2 + 4 * g];
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
    // Per-split results, then join the head's splits and merge this split's
    // share of the rows.
    const size_t head_base = (size_t)h * S * p.Mp;
    const size_t split_base = head_base + (size_t)s * p.Mp;
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      const int rb = wave + 4 * r;
      if (rb >= MB) continue;
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
      __hip_atomic_fetch_add(&p.head_cnt[h], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (!wait_at_least(sy, &p.head_cnt[h], S * (layer + 1))) return false;

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
    bf16* obase = p.o + (size_t)layer * p.Mp * d;
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
      st_coherent_bf2(obase + (size_t)i * d + h * DH + dd, o0, o1);
    }
    __syncthreads();
  }
  return true;
}

// ------------------------------------------------------------------ embed

__device__ __forceinline__ void embed_phase(const PassParams& p, const TreeArgs& tree) {
  __shared__ int par_s[128];
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
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int m = blockIdx.x; m < p.Mp; m += p.G) {
    const bool valid = m < p.n;
    const bf16* row = E + (size_t)(valid ? tree.tok[m] : 0) * p.d;
    for (int t = wave; t < p.d_tiles; t += kWaves) {
      const int c = 64 * t + lane;
      const float v = valid ? bf2f(row[c]) : 0.0f;
      st_coherent(&p.x[(size_t)m * p.d + c], v);
      const float s = wave_sum(v * v);
      if (lane == 0) st_coherent(&p.ssq[(size_t)t * p.Mp + m], s);
    }
  }
}

// ------------------------------------------------------------------ kernel

template <int MB, int DH>
__global__ __launch_bounds__(kThreads, 1) void pass_kernel(const PassParams p, const TreeArgs tree) {
  constexpr int D = MB <= 2 ? 4 : (MB <= 4 ? 3 : 2);
  __shared__ __attribute__((aligned(16))) char attn_lds[AttnLds<MB, DH>::BYTES];
  __shared__ PassLds<MB> lds;
  __shared__ int flag;
  const Sync sy{p.bar, p.status, p.spin_limit, &flag,
                p.trace != nullptr && (int)blockIdx.x < kTraceWgs
                    ? p.trace + (size_t)blockIdx.x * (2 + 5 * p.L) * 6
                    : nullptr};
  const int G = p.G;
  const size_t xsz = (size_t)p.Mp * p.d, ssz = (size_t)p.d_tiles * p.Mp;
  int phase = 0;
  bool ok = true;

  embed_phase(p, tree);
  grid_arrive(sy, phase);
  ++phase;

  for (int l = 0; l < p.L && ok; ++l) {
    const char* lw = p.packed + p.layer0 + (long long)l * p.layer_bytes;
    const float* x_a = p.x + (size_t)(2 * l) * xsz;       // layer input
    float* x_b = p.x + (size_t)(2 * l + 1) * xsz;         // after attention
    float* x_c = p.x + (size_t)(2 * l + 2) * xsz;         // after feed-forward
    const float* ss_a = p.ssq + (size_t)(2 * l) * ssz;
    float* ss_b = p.ssq + (size_t)(2 * l + 1) * ssz;
    float* ss_c = p.ssq + (size_t)(2 * l + 2) * ssz;
    bf16* q_l = p.q + (size_t)l * p.Mp * p.d;
    bf16* o_l = p.o + (size_t)l * p.Mp * p.d;
    bf16* h_l = p.h + (size_t)l * p.Mp * p.Fp;
    const size_t kv_layer = (size_t)p.H * p.cap * p.Dh;

    {  // QKV
      GemmDesc g{(const bf16x8*)(lw + p.o_qkv), p.qkv_tiles, p.ks_d, nullptr, 0, x_a, ss_a,
                 (const bf16*)(lw + p.o_attn_norm)};
      EpiQkv e{q_l, p.k_cache + (size_t)l * kv_layer, p.v_cache + (size_t)l * kv_layer, p.tree + 384};
      ok = gemm_phase<MB, PRO_NORM, EPI_QKV, D>(p, g, sy, G * phase, lds, l, &e);
      if (!ok) break;
      grid_arrive(sy, phase);
      ++phase;
    }
    ok = attn_phase<MB, DH>(p, l, sy, G * phase, attn_lds);
    if (!ok) break;
    grid_arrive(sy, phase);
    ++phase;
    {  // O projection + residual
      GemmDesc g{(const bf16x8*)(lw + p.o_o), p.d_tiles, p.ks_d, o_l, p.d, nullptr, nullptr, nullptr};
      EpiResid e{x_a, x_b, ss_b};
      ok = gemm_phase<MB, PRO_BF16, EPI_RESID, D>(p, g, sy, G * phase, lds, l, &e);
      if (!ok) break;
      grid_arrive(sy, phase);
      ++phase;
    }
    {  // gate/up + SwiGLU
      GemmDesc g{(const bf16x8*)(lw + p.o_gu), p.gu_tiles, p.ks_d, nullptr, 0, x_b, ss_b,
                 (const bf16*)(lw + p.o_ffn_norm)};
      EpiSwiglu e{h_l};
      ok = gemm_phase<MB, PRO_NORM, EPI_SWIGLU, D>(p, g, sy, G * phase, lds, l, &e);
      if (!ok) break;
      grid_arrive(sy, phase);
      ++phase;
    }
    {  // down projection + residual
      GemmDesc g{(const bf16x8*)(lw + p.o_down), p.d_tiles, p.ks_f, h_l, p.Fp, nullptr, nullptr, nullptr};
      EpiResid e{x_b, x_c, ss_c};
      ok = gemm_phase<MB, PRO_BF16, EPI_RESID, D>(p, g, sy, G * phase, lds, l, &e);
      if (!ok) break;
      grid_arrive(sy, phase);
      ++phase;
    }
  }
  if (ok) {  // final norm + LM head + argmax + accept walk
    GemmDesc g{(const bf16x8*)(p.packed + p.o_lm), p.v_tiles, p.ks_d, nullptr, 0,
               p.x + (size_t)(2 * p.L) * xsz, p.ssq + (size_t)(2 * p.L) * ssz,
               (const bf16*)(p.packed + p.o_final_norm)};
    EpiLogits e{p.logits, p.row_lo};
    if (gemm_phase<MB, PRO_NORM, EPI_LOGITS, D>(p, g, sy, G * phase, lds, p.L, &e))
      trace_mark(sy, phase, 2);
  }
  // Leave the pass: the last workgroup out resets the barrier and join counters.
  if (arrive_last(p.exit_cnt, G, &flag)) {
    if (threadIdx.x < kBarSlots)
      __hip_atomic_store(p.bar + threadIdx.x * kBarStride, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    for (int h = threadIdx.x; h < p.H; h += kThreads)
      __hip_atomic_store(&p.head_cnt[h], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

template <int MB, int DH>
hipError_t launch_pass_mb(const PassParams& p, const TreeArgs& tree, hipStream_t st) {
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

hipError_t launch_pass(int mb, const PassParams& p, const TreeArgs& tree, hipStream_t st) {
#define LLMCAD_PASS_CASE(M)                                                 \
  case M:                                                                   \
    return p.Dh == 128 ? launch_pass_mb<M, 128>(p, tree, st)                \
                       : launch_pass_mb<M, 64>(p, tree, st);
  switch (mb) {
    LLMCAD_PASS_CASE(1)
    LLMCAD_PASS_CASE(2)
    LLMCAD_PASS_CASE(3)
    LLMCAD_PASS_CASE(4)
    LLMCAD_PASS_CASE(5)
    LLMCAD_PASS_CASE(6)
    LLMCAD_PASS_CASE(7)
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
    LLMCAD_OCC_CASE(5)
    LLMCAD_OCC_CASE(6)
    LLMCAD_OCC_CASE(7)
    LLMCAD_OCC_CASE(8)
    default:
      return 0;
  }
#undef LLMCAD_OCC_CASE
}

}  // namespace llmcad
