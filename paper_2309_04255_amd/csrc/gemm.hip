// Skinny GEMM for the verification pass: Y[n x N] = A[n x K] * W^T with n <= 128
// tree nodes and W streamed once from HBM in packed MFMA-fragment order.
//
// Why this shape: one pass visits every weight once for all n nodes (the
// non-autoregressive verification of §3.2), so the work is bound by reading
// W; n is the M dimension of a 16x16x32 bf16 MFMA (rows padded to 16).
//
// Work decomposition
//  - A workgroup (4 waves) owns one 64-column tile and one contiguous run of
//    k-steps (split-K); its 4 waves take interleaved k-steps, so together they
//    read the run as consecutive 4 KiB blocks.  Each wave keeps D k-steps of
//    loads in flight (register double/quad buffering).
//  - Wave partials are summed in LDS in a fixed order (wave 0, 1, 2, 3); with
//    split-K each workgroup stores its partial tile, and the last workgroup to
//    arrive at the tile's counter sums the partials in split order.  Results
//    are therefore bit-reproducible run to run.
//  - The tile's epilogue runs in that last workgroup.
//
// Prologues (how the A operand is formed)
//  PRO_BF16  A is a bf16 activation matrix (attention output, SwiGLU product).
//  PRO_NORM  A = bf16(x * rstd(row) * gain) from the fp32 residual stream:
//            RMSNorm fused into the load; rstd comes from per-tile sums of
//            squares left by the producer of x, summed in a fixed order.
// Epilogues
//  EPI_QKV     rotary embedding at the node's position, q to the workspace,
//              k/v into the node's KV-cache slot (prefix_len + node).
//  EPI_RESID   x += tile, plus the tile's per-row sum of squares of the new x.
//  EPI_SWIGLU  h = bf16(silu(gate) * up).
//  EPI_LOGITS  fp32 logits, per-tile row argmax; the last tile to finish
//              reduces the argmax over tiles and runs the accept walk.
#include <math.h>

#include "device.h"
#include "kernels.h"
#include "layout.h"

namespace llmcad {

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

template <int MB, int PRO, int EPI, int D>
__global__ __launch_bounds__(256) void gemm_kernel(const GemmParams p) {
  constexpr int ROWS = MB * 16;
  constexpr int TS = 64 + 4;  // LDS row stride in floats
  __shared__ float tileS[ROWS][TS];
  __shared__ int flag;
  __shared__ int reach[EPI == EPI_LOGITS ? kMaxNodes : 1];
  __shared__ int amax_s[EPI == EPI_LOGITS ? kMaxNodes : 1];

  const int tile = blockIdx.x / p.ksplit;
  const int split = blockIdx.x - tile * p.ksplit;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int lrow = lane & 15, kg = lane >> 4;
  const int s_begin = (int)((long)split * p.ksteps / p.ksplit);
  const int s_end = (int)((long)(split + 1) * p.ksteps / p.ksplit);
  const int s0 = s_begin + wave;
  const int ns = s0 < s_end ? (s_end - s0 + 3) / 4 : 0;  // k-steps of this wave

  float rstd[MB];
  if constexpr (PRO == PRO_NORM) {
    // rstd(row) from the per-tile sums of squares: the block's threads split
    // the tiles into CH contiguous chunks, then the chunks are added in
    // order, so every workgroup forms the same value.
    constexpr int CH = 256 / ROWS;
    __shared__ float part_ss[CH][ROWS];
    if (threadIdx.x < CH * ROWS) {
      const int r = threadIdx.x % ROWS, c = threadIdx.x / ROWS;
      const int t0 = c * p.ssq_tiles / CH, t1 = (c + 1) * p.ssq_tiles / CH;
      float ss = 0.0f;
      int t = t0;
      for (; t + 4 <= t1; t += 4) {
        const float v0 = p.ssq[(size_t)t * p.Mp + r], v1 = p.ssq[(size_t)(t + 1) * p.Mp + r];
        const float v2 = p.ssq[(size_t)(t + 2) * p.Mp + r], v3 = p.ssq[(size_t)(t + 3) * p.Mp + r];
        ss += v0;
        ss += v1;
        ss += v2;
        ss += v3;
      }
      for (; t < t1; ++t) ss += p.ssq[(size_t)t * p.Mp + r];
      part_ss[c][r] = ss;
    }
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) {
      const int row = 16 * rb + lrow;
      float ss = 0.0f;
#pragma unroll
      for (int c = 0; c < CH; ++c) ss += part_ss[c][row];
      rstd[rb] = 1.0f / sqrtf(ss * p.inv_d + p.eps);
    }
  }

  f32x4 acc[MB][4];
#pragma unroll
  for (int rb = 0; rb < MB; ++rb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[rb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (ns > 0) {
    const bf16x8* __restrict__ wt = (const bf16x8*)p.w + (size_t)tile * p.ksteps * 256 + lane;
    bf16x8 bw[D][4];
    AStage<MB, PRO> as[D];

    auto load = [&](int slot, int i) {
      const int s = s0 + 4 * i;
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) bw[slot][nb] = wt[(size_t)s * 256 + nb * 64];
      const int k = 32 * s + 8 * kg;
      if constexpr (PRO == PRO_BF16) {
        const bf16* A = (const bf16*)p.a;
#pragma unroll
        for (int rb = 0; rb < MB; ++rb)
          as[slot].a[rb] = *(const bf16x8*)(A + (size_t)(16 * rb + lrow) * p.lda + k);
      } else {
#pragma unroll
        for (int rb = 0; rb < MB; ++rb) {
          const float* xr = p.x + (size_t)(16 * rb + lrow) * p.d + k;
          as[slot].x[rb][0] = *(const float4*)xr;
          as[slot].x[rb][1] = *(const float4*)(xr + 4);
        }
        as[slot].g = *(const bf16x8*)((const bf16*)p.gain + k);
      }
    };

    auto compute = [&](int slot) {
#pragma unroll
      for (int rb = 0; rb < MB; ++rb) {
        bf16x8 a;
        if constexpr (PRO == PRO_BF16) {
          a = as[slot].a[rb];
        } else {
          const float xs[8] = {as[slot].x[rb][0].x, as[slot].x[rb][0].y, as[slot].x[rb][0].z,
                               as[slot].x[rb][0].w, as[slot].x[rb][1].x, as[slot].x[rb][1].y,
                               as[slot].x[rb][1].z, as[slot].x[rb][1].w};
#pragma unroll
          for (int e = 0; e < 8; ++e) a[e] = f2bf(xs[e] * rstd[rb] * bf2f(as[slot].g[e]));
        }
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) acc[rb][nb] = mfma16x16x32(a, bw[slot][nb], acc[rb][nb]);
      }
    };

    // Loads are issued unconditionally (clamped to the last step) so that the
    // number of loads in flight is the same on every path.
#pragma unroll
    for (int u = 0; u < D; ++u) load(u, u < ns ? u : ns - 1);
    for (int i = 0; i < ns; i += D) {
#pragma unroll
      for (int u = 0; u < D; ++u) {
        if (i + u < ns) compute(u);
        const int nx = i + u + D;
        load(u, nx < ns ? nx : ns - 1);
      }
    }
  }

  // Sum the four waves' partial tiles in LDS, in wave order.
  for (int w = 0; w < 4; ++w) {
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

  if (p.ksplit > 1) {
    float* mine = p.part + (size_t)blockIdx.x * ROWS * 64;
    for (int idx = 2 * threadIdx.x; idx < ROWS * 64; idx += 512)
      st_coherent2(mine + idx, tileS[idx >> 6][idx & 63], tileS[idx >> 6][(idx & 63) + 1]);
    if (!arrive_last(&p.counters[tile], p.ksplit, &flag)) return;
    const float* base = p.part + (size_t)tile * p.ksplit * ROWS * 64;
    for (int idx = 2 * threadIdx.x; idx < ROWS * 64; idx += 512) {
      float s0 = 0.0f, s1 = 0.0f;
      int sp = 0;
      for (; sp + 4 <= p.ksplit; sp += 4) {  // four loads in flight, sums in split order
        float2 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = ld_coherent2(base + (size_t)(sp + u) * ROWS * 64 + idx);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          s0 += v[u].x;
          s1 += v[u].y;
        }
      }
      for (; sp < p.ksplit; ++sp) {
        const float2 v = ld_coherent2(base + (size_t)sp * ROWS * 64 + idx);
        s0 += v.x;
        s1 += v.y;
      }
      tileS[idx >> 6][idx & 63] = s0;
      tileS[idx >> 6][(idx & 63) + 1] = s1;
    }
    __syncthreads();
  }

  // ---------------------------------------------------------------- epilogues
  if constexpr (EPI == EPI_QKV) {
    const int tiles_per_head = p.Dh / 64;
    const int per_part = p.H * tiles_per_head;
    const int part = tile / per_part, rr = tile % per_part;
    const int h = rr / tiles_per_head, b = rr % tiles_per_head;
    const int half = p.Dh / 2;
    const int jj = 32 * b + (lane & 31);  // rotary pair index in [0, Dh/2)
    const int j = lane < 32 ? jj : half + jj;
    const float inv_freq = exp2f(-(2.0f * (float)jj / (float)p.Dh) * p.log2_theta);
    const int d = p.H * p.Dh;
    for (int r = wave; r < p.n; r += 4) {
      const float v = tileS[r][lane];
      float out = v;
      if (part < 2) {
        const float partner = tileS[r][lane ^ 32];
        float sn, cs;
        sincosf((float)p.pos[r] * inv_freq, &sn, &cs);
        out = lane < 32 ? v * cs - partner * sn : v * cs + partner * sn;
      }
      const bf16 ob = f2bf(out);
      if (part == 0) {
        ((bf16*)p.q_out)[(size_t)r * d + h * p.Dh + j] = ob;
      } else {
        bf16* cache = (bf16*)(part == 1 ? p.k_cache : p.v_cache);
        cache[((size_t)h * p.cap + p.prefix_len + r) * p.Dh + j] = ob;
      }
    }
  } else if constexpr (EPI == EPI_RESID) {
    const int col = 64 * tile + lane;
    for (int r = wave; r < ROWS; r += 4) {
      float xn = 0.0f;
      if (r < p.n) {
        float* xp = p.x_out + (size_t)r * p.d + col;
        xn = *xp + tileS[r][lane];
        *xp = xn;
      }
      const float s = wave_sum(xn * xn);
      if (lane == 0) p.ssq_out[(size_t)tile * p.Mp + r] = s;
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    const int c = lane & 31;
    for (int r = wave; r < p.n; r += 4) {
      if (lane < 32) {
        const float g = tileS[r][c], u = tileS[r][32 + c];
        const float hval = g / (1.0f + expf(-g)) * u;
        ((bf16*)p.h_out)[(size_t)r * p.ldh + 32 * tile + c] = f2bf(hval);
      }
    }
  } else {  // EPI_LOGITS
    const int col = 64 * tile + lane;
    for (int r = wave; r < ROWS; r += 4) {
      const bool valid = r < p.n && col < p.V;
      const float v = tileS[r][lane];
      if (valid && p.logits != nullptr && r >= p.row_lo)
        p.logits[(size_t)(r - p.row_lo) * p.V + col] = v;
      float mv = valid ? v : -INFINITY;
      int mi = valid ? col : 0x7fffffff;
      wave_argmax(mv, mi);
      if (lane == 0) {
        st_coherent(&p.lm_val[(size_t)tile * p.Mp + r], mv);
        st_coherent(&p.lm_idx[(size_t)tile * p.Mp + r], mi);
      }
    }
    if (!arrive_last(p.lm_counter, p.tiles, &flag)) return;
    // Greedy target token per node: argmax over all tiles (lowest column on ties).
    for (int r = wave; r < p.n; r += 4) {
      float mv = -INFINITY;
      int mi = 0x7fffffff;
      for (int t0 = 0; t0 < p.tiles; t0 += 4 * 64) {  // four loads per lane in flight
        float v[4];
        int ix[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int t = t0 + 64 * u + lane;
          v[u] = t < p.tiles ? ld_coherent(&p.lm_val[(size_t)t * p.Mp + r]) : -INFINITY;
          ix[u] = t < p.tiles ? ld_coherent(&p.lm_idx[(size_t)t * p.Mp + r]) : 0x7fffffff;
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
        amax_s[r] = mi;
      }
    }
    __syncthreads();
    // Accept walk (§3.2): node i is reachable when its parent is reachable and
    // its draft token equals the target's token after its parent; the result
    // is the deepest reachable node (lowest index among equally deep ones).
    if (threadIdx.x == 0) {
      int best = 0, best_depth = 0;
      reach[0] = 1;
      for (int i = 1; i < p.n; ++i) {
        const int par = p.tree_parent[i];
        const int ok = reach[par] && (p.tree_tok[i] == amax_s[par]);
        reach[i] = ok;
        const int dep = p.tree_depth[i];
        if (ok && dep > best_depth) {
          best = i;
          best_depth = dep;
        }
      }
      for (int k = 0; k < p.n; ++k) p.path[k] = -1;
      for (int i = best; i >= 0; i = p.tree_parent[i]) p.path[p.tree_depth[i]] = i;
      *p.accept_len = best_depth;
      *p.next_token = amax_s[best];
    }
  }
}

template <int MB, int PRO, int EPI>
static hipError_t launch_mb(const GemmParams& p, hipStream_t st) {
  constexpr int D = MB <= 2 ? 4 : (MB <= 4 ? 3 : 2);
  const dim3 grid(p.tiles * p.ksplit), block(256);
  gemm_kernel<MB, PRO, EPI, D><<<grid, block, 0, st>>>(p);
  return hipGetLastError();
}

template <int PRO, int EPI>
static hipError_t launch_pe(int mb, const GemmParams& p, hipStream_t st) {
  switch (mb) {
    case 1: return launch_mb<1, PRO, EPI>(p, st);
    case 2: return launch_mb<2, PRO, EPI>(p, st);
    case 3: return launch_mb<3, PRO, EPI>(p, st);
    case 4: return launch_mb<4, PRO, EPI>(p, st);
    case 5: return launch_mb<5, PRO, EPI>(p, st);
    case 6: return launch_mb<6, PRO, EPI>(p, st);
    case 7: return launch_mb<7, PRO, EPI>(p, st);
    case 8: return launch_mb<8, PRO, EPI>(p, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm(int pro, int epi, int mb, const GemmParams& p, hipStream_t st) {
  if (pro == PRO_NORM && epi == EPI_QKV) return launch_pe<PRO_NORM, EPI_QKV>(mb, p, st);
  if (pro == PRO_BF16 && epi == EPI_RESID) return launch_pe<PRO_BF16, EPI_RESID>(mb, p, st);
  if (pro == PRO_NORM && epi == EPI_SWIGLU) return launch_pe<PRO_NORM, EPI_SWIGLU>(mb, p, st);
  if (pro == PRO_NORM && epi == EPI_LOGITS) return launch_pe<PRO_NORM, EPI_LOGITS>(mb, p, st);
  return hipErrorInvalidValue;
}

}  // namespace llmcad
