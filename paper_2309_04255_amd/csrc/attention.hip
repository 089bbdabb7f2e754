// Tree-masked attention for one verification pass.
//
// Node i (query row) attends to key positions [0, prefix_len) and to the
// cache slots prefix_len + j of its ancestors-or-self j: the tree masking
// table of §3.2 ("Tree decoder"), one row per node, held as a 128-bit set.
//
// Grid: (head, split); a split is a run of 64-position chunks of
// [0, prefix_len + n).  Per chunk, the workgroup stages K (row-major) and V
// (transposed) in LDS with 16-byte global loads; each wave owns up to two
// 16-row query blocks and runs an online softmax:
//   S^T = K q^T     (MFMA, A = K rows from LDS, B = q fragment in registers)
//   P   = exp2(S * log2(e)/sqrt(Dh) - m), masked entries 0, split P = Phi + Plo
//         into two bf16 parts so the product keeps ~16 bits of P
//   O^T += V^T Phi^T + V^T Plo^T  (MFMA, A = V^T from LDS, B = P straight from
//         the S result)
// The S result leaves lane l holding row (l % 16) and keys 4(l/16)+e of each
// 16-key block; the PV product takes its k-slots in exactly that order, so P
// never goes through LDS, and the output lands in the same rows per lane.
// Each split writes (max, sum, unnormalised O) per row; the last workgroup
// of a head merges the splits in split order and writes bf16 o.
#include <math.h>

#include "device.h"
#include "kernels.h"
#include "layout.h"

namespace llmcad {

template <int RPW, int DH>
__global__ __launch_bounds__(256) void attn_kernel(const AttnParams p) {
  constexpr int CH = kAttnChunk;   // 64 key positions per step
  constexpr int KSTEPS = DH / 32;  // MFMA k-steps over the head dimension
  constexpr int DB = DH / 16;      // 16-wide output column blocks
  constexpr int KST = DH + 8;      // LDS row stride of K (bf16)
  constexpr int VST = CH + 8;      // LDS row stride of V^T (bf16)
  // LDS: the K and V^T tiles of the chunk loop, reused by the split merge.
  constexpr int KS_BYTES = CH * KST * 2, VT_BYTES = DH * VST * 2;
  constexpr int MERGE_BYTES = 2 * kAttnMaxSplits * kMaxNodes * 4;
  constexpr int LDS_BYTES = KS_BYTES + VT_BYTES > MERGE_BYTES ? KS_BYTES + VT_BYTES : MERGE_BYTES;
  __shared__ __attribute__((aligned(16))) char lds_raw[LDS_BYTES];
  __shared__ int flag;
  bf16* Ks = reinterpret_cast<bf16*>(lds_raw);
  bf16* Vt = reinterpret_cast<bf16*>(lds_raw + KS_BYTES);

  const int h = blockIdx.x / p.splits, sp = blockIdx.x % p.splits;
  const int c_begin = sp * p.nchunks / p.splits, c_end = (sp + 1) * p.nchunks / p.splits;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int li = lane & 15, g = lane >> 4;
  const int MB = p.Mp / 16;
  const int total = p.prefix_len + p.n;
  const int d = p.H * DH;
  const bf16* __restrict__ kc = (const bf16*)p.k_cache + (size_t)h * p.cap * DH;
  const bf16* __restrict__ vc = (const bf16*)p.v_cache + (size_t)h * p.cap * DH;

  bf16x8 qf[RPW][KSTEPS];
  uint32_t anc[RPW][4];
  float m_run[RPW], l_run[RPW];
  f32x4 oacc[RPW][DB];
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    const int rb = wave + 4 * r;
    const int row = 16 * (rb < MB ? rb : 0) + li;
    const bf16* qr = (const bf16*)p.q + (size_t)row * d + h * DH;
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) qf[r][ks] = *(const bf16x8*)(qr + 32 * ks + 8 * g);
#pragma unroll
    for (int w = 0; w < 4; ++w) anc[r][w] = p.anc[row * 4 + w];
    m_run[r] = -INFINITY;
    l_run[r] = 0.0f;
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[r][db] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  for (int c = c_begin; c < c_end; ++c) {
    const int p0 = c * CH;
    __syncthreads();  // the previous chunk's LDS reads are done
    for (int idx = threadIdx.x; idx < CH * DH / 8; idx += 256) {
      const int j = idx / (DH / 8), dc = (idx % (DH / 8)) * 8;
      const int pos = p0 + j;
      bf16x8 kv, vv;
      if (pos < total) {
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
      // Mask (prefix always visible; tree slots only for ancestors-or-self)
      // and scale into the log2 domain.
      float mx = -INFINITY;
#pragma unroll
      for (int jb = 0; jb < 4; ++jb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int pos = p0 + 16 * jb + 4 * g + e;
          const int t = pos - p.prefix_len;
          const bool vis = pos < p.prefix_len ||
                           (t < p.n && ((anc[r][t >> 5] >> (t & 31)) & 1u));
          const float s = vis ? sc[jb][e] * p.scale_log2 : -INFINITY;
          sc[jb][e] = s;
          mx = fmaxf(mx, s);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
      mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
      const float m_new = fmaxf(m_run[r], mx);
      const float m_use = (m_new == -INFINITY) ? 0.0f : m_new;
      const float alpha = exp2f(m_run[r] - m_use);
      // p = hi + lo with both halves bf16: the PV product then carries p to
      // about 16 significant bits although the matrix cores take bf16.
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
          const bf16x4 lo = *(const bf16x4*)vrow;
          const bf16x4 hi = *(const bf16x4*)(vrow + 16);
          bf16x8 av;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            av[e] = lo[e];
            av[4 + e] = hi[e];
          }
          oacc[r][db] = mfma16x16x32(av, bph, oacc[r][db]);
          oacc[r][db] = mfma16x16x32(av, bpl, oacc[r][db]);
        }
      }
    }
  }

  // Per-split results: lane l holds O[row 16 rb + l%16][16 db + 4 (l/16) + e].
  const size_t split_base = ((size_t)h * p.splits + sp) * p.Mp;
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    const int rb = wave + 4 * r;
    if (rb >= MB) continue;
    const int row = 16 * rb + li;
    if (g == 0) st_coherent2(&p.part_ml[(split_base + row) * 2], m_run[r], l_run[r]);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      float* dst = &p.part_o[(split_base + row) * DH + 16 * db + 4 * g];
      st_coherent2(dst, oacc[r][db][0], oacc[r][db][1]);
      st_coherent2(dst + 2, oacc[r][db][2], oacc[r][db][3]);
    }
  }

  if (!arrive_last(&p.counters[h], p.splits, &flag)) return;

  // Merge the splits of head h in split order: per-row weights first (in
  // LDS), then every output element as a weighted sum of the split outputs.
  float (*wgt)[kMaxNodes] = reinterpret_cast<float (*)[kMaxNodes]>(lds_raw);
  float (*lsum)[kMaxNodes] = wgt + kAttnMaxSplits;
  const int S = p.splits;
  const size_t head_base = (size_t)h * S * p.Mp;
  for (int idx = threadIdx.x; idx < S * p.n; idx += 256) {
    const int s = idx / p.n, i = idx % p.n;
    const float2 ml = ld_coherent2(&p.part_ml[(head_base + (size_t)s * p.Mp + i) * 2]);
    wgt[s][i] = ml.x;
    lsum[s][i] = ml.y;
  }
  __syncthreads();
  if (threadIdx.x < p.n) {
    const int i = threadIdx.x;
    float M = -INFINITY;
    for (int s = 0; s < S; ++s) M = fmaxf(M, wgt[s][i]);
    float L = 0.0f;
    for (int s = 0; s < S; ++s) {
      const float w = exp2f(wgt[s][i] - M);
      wgt[s][i] = w;
      L += lsum[s][i] * w;
    }
    const float inv = 1.0f / L;
    for (int s = 0; s < S; ++s) wgt[s][i] *= inv;
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < p.n * (DH / 2); idx += 256) {
    const int i = idx / (DH / 2), dd = 2 * (idx % (DH / 2));
    float o0 = 0.0f, o1 = 0.0f;
    int s = 0;
    for (; s + 4 <= S; s += 4) {  // four loads in flight, sums in split order
      float2 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        v[u] = ld_coherent2(&p.part_o[(head_base + (size_t)(s + u) * p.Mp + i) * DH + dd]);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        o0 += v[u].x * wgt[s + u][i];
        o1 += v[u].y * wgt[s + u][i];
      }
    }
    for (; s < S; ++s) {
      const float2 v = ld_coherent2(&p.part_o[(head_base + (size_t)s * p.Mp + i) * DH + dd]);
      o0 += v.x * wgt[s][i];
      o1 += v.y * wgt[s][i];
    }
    bf16* dst = (bf16*)p.o_out + (size_t)i * d + h * DH + dd;
    dst[0] = f2bf(o0);
    dst[1] = f2bf(o1);
  }
}

template <int RPW>
static hipError_t launch_rpw(const AttnParams& p, hipStream_t st) {
  const dim3 grid(p.H * p.splits), block(256);
  if (p.Dh == 128)
    attn_kernel<RPW, 128><<<grid, block, 0, st>>>(p);
  else if (p.Dh == 64)
    attn_kernel<RPW, 64><<<grid, block, 0, st>>>(p);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attention(int mb, const AttnParams& p, hipStream_t st) {
  return mb > 4 ? launch_rpw<2>(p, st) : launch_rpw<1>(p, st);
}

}  // namespace llmcad
