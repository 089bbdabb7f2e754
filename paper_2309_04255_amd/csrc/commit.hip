// Rollback after a verification pass (§3.2 "Token tree verification and
// rectification": the tree is rolled back to its verified sequence, which
// becomes the input of the next generation step).
//
// The pass wrote node i's keys and values to cache slot prefix_len + i, at
// the position the node keeps if accepted (prefix_len + its depth).  The
// accepted nodes are path[0] = 0 (the root), path[1..len], one per depth, so
// committing them is a move of slot prefix_len + path[k] to prefix_len + k for
// every layer and head.  path[k] >= k, and a slot written here can be the
// source of a row with a smaller k, so each workgroup (one (layer, head) pair)
// reads all its accepted rows into LDS before it writes any.
#include "device.h"
#include "kernels.h"

namespace llmcad {

namespace {

__global__ __launch_bounds__(256) void commit_kernel(bf16* __restrict__ k_cache, bf16* __restrict__ v_cache,
                                                     int cap, int prefix_len, const int* __restrict__ path,
                                                     const int* __restrict__ accept_len, int n, int dh) {
  extern __shared__ bf16x8 rows[];  // [2][len + 1][dh / 8]: K rows, then V rows
  const int len = ldg(accept_len);
  if (len < 1 || len >= n) return;  // nothing moves (or not the output of a pass over n nodes)
  const int cpr = dh / 8;            // 16-byte chunks per row
  const int items = (len + 1) * cpr;
  const size_t base = (size_t)blockIdx.x * cap * dh;  // this (layer, head)'s rows
  for (int e = threadIdx.x; e < items; e += blockDim.x) {
    const int k = e / cpr, c = e % cpr;
    const int src = ldg(path + k);
    const bool ok = src >= k && src < n;
    const size_t at = base + (size_t)(prefix_len + (ok ? src : k)) * dh + 8 * c;
    rows[e] = ldg((const bf16x8*)(k_cache + at));
    rows[items + e] = ldg((const bf16x8*)(v_cache + at));
  }
  __syncthreads();
  for (int e = threadIdx.x; e < items; e += blockDim.x) {
    const int k = e / cpr, c = e % cpr;
    const int src = ldg(path + k);
    if (src == k || src < k || src >= n) continue;  // in place already (or an invalid entry: left alone)
    const size_t at = base + (size_t)(prefix_len + k) * dh + 8 * c;
    stg((bf16x8*)(k_cache + at), rows[e]);
    stg((bf16x8*)(v_cache + at), rows[items + e]);
  }
}

}  // namespace

hipError_t launch_commit(void* k_cache, void* v_cache, int layers_heads, int cap, int prefix_len, const int* path,
                         const int* accept_len, int n, int dh, hipStream_t st) {
  const size_t lds = (size_t)2 * n * dh * sizeof(bf16);
  commit_kernel<<<dim3(layers_heads), dim3(256), lds, st>>>((bf16*)k_cache, (bf16*)v_cache, cap, prefix_len, path,
                                                             accept_len, n, dh);
  return hipGetLastError();
}

}  // namespace llmcad
