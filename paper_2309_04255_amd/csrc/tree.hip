// Tree preparation and token embedding: the first step of a verification pass.
//
// From parent[] (topological order, parent[0] = -1) every node's depth, its
// position (prefix_len + depth: a node continues its own branch, not the
// order nodes were drafted in) and its ancestor-or-self bit set are derived;
// the bit set is the row of the tree masking table (§3.2 "Tree decoder": a
// token sees only earlier positions of its own branch).  The residual stream
// starts as the nodes' embedding rows, and per-64-column sums of squares are
// written for the first RMSNorm.
#include "device.h"
#include "kernels.h"

namespace llmcad {

// ws_tree layout: int32 tok[128] | parent[128] | depth[128] | pos[128] | uint32 anc[128][4]
__global__ __launch_bounds__(256) void embed_kernel(TreeArgs tree, int n, int Mp, int d,
                                                    int prefix_len, const bf16* __restrict__ E,
                                                    int* __restrict__ ws_tree,
                                                    float* __restrict__ x,
                                                    float* __restrict__ ssq) {
  const int m = blockIdx.x;
  __shared__ int par_s[128];
  if (m == 0) {
    if (threadIdx.x < 128) par_s[threadIdx.x] = threadIdx.x < n ? tree.parent[threadIdx.x] : -1;
    __syncthreads();
  }
  if (m == 0 && threadIdx.x < 128) {
    // Each node walks its own ancestor chain (all nodes in parallel).
    const int i = threadIdx.x;
    int dep = 0;
    uint32_t a[4] = {0u, 0u, 0u, 0u};
    if (i < n) {
      for (int j = i; j >= 0; j = par_s[j]) {
        a[j >> 5] |= 1u << (j & 31);
        ++dep;
      }
      --dep;
    }
    ws_tree[i] = i < n ? tree.tok[i] : 0;
    ws_tree[128 + i] = par_s[i];
    ws_tree[256 + i] = dep;
    ws_tree[384 + i] = prefix_len + dep;
    uint32_t* anc = (uint32_t*)(ws_tree + 512);
#pragma unroll
    for (int w = 0; w < 4; ++w) anc[i * 4 + w] = a[w];
  }
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const bool valid = m < n;
  const bf16* row = E + (size_t)(valid ? tree.tok[m] : 0) * d;
  float* xr = x + (size_t)m * d;
  for (int t = wave; t < d / 64; t += 4) {
    const int c = 64 * t + lane;
    const float v = valid ? bf2f(row[c]) : 0.0f;
    xr[c] = v;
    const float s = wave_sum(v * v);
    if (lane == 0) ssq[(size_t)t * Mp + m] = s;
  }
}

hipError_t launch_embed(const TreeArgs& tree, int n, int Mp, int d, int prefix_len,
                        const void* tok_embed, void* ws_tree, float* x, float* ssq,
                        hipStream_t st) {
  embed_kernel<<<dim3(Mp), dim3(256), 0, st>>>(tree, n, Mp, d, prefix_len, (const bf16*)tok_embed,
                                                (int*)ws_tree, x, ssq);
  return hipGetLastError();
}

}  // namespace llmcad
