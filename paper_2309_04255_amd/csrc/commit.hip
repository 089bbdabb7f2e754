// Rollback after a verification pass (§3.2 "Token tree verification and
// rectification": the tree is rolled back to its verified sequence, which
// becomes the input of the next generation step).
//
// The pass wrote node i's keys and values to cache slot prefix_len + i (K
// row-major per head, V transposed per head), at
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
  // LDS: the K rows [len + 1][dh / 8] (16-byte pieces), then the V entries
  // [dh][len + 1] (the V cache is transposed per head: a slot is one entry of
  // each of the head's dh rows)
  extern __shared__ bf16x8 rows[];
  const int len = ldg(accept_len);
  if (len < 1 || len >= n) return;  // nothing moves (or not the output of a pass over n nodes)
  const int cpr = dh / 8;            // 16-byte pieces per K row
  const int kitems = (len + 1) * cpr, vitems = (len + 1) * dh;
  bf16* vents = (bf16*)(rows + kitems);
  const size_t base = (size_t)blockIdx.x * cap * dh;  // this (layer, head)'s K rows, and its V^T rows
  auto source = [&](int k) {
    const int src = ldg(path + k);
    return src >= k && src < n ? src : k;  // (an invalid entry reads its own slot: left alone)
  };
  for (int e = threadIdx.x; e < kitems; e += blockDim.x) {
    const int k = e / cpr, c = e % cpr;
    rows[e] = ldg((const bf16x8*)(k_cache + base + (size_t)(prefix_len + source(k)) * dh + 8 * c));
  }
  for (int e = threadIdx.x; e < vitems; e += blockDim.x) {
    const int dim = e / (len + 1), k = e % (len + 1);
    vents[e] = ldg(v_cache + base + (size_t)dim * cap + prefix_len + source(k));
  }
  __syncthreads();
  for (int e = threadIdx.x; e < kitems; e += blockDim.x) {
    const int k = e / cpr, c = e % cpr;
    if (source(k) == k) continue;  // in place already
    stg((bf16x8*)(k_cache + base + (size_t)(prefix_len + k) * dh + 8 * c), rows[e]);
  }
  for (int e = threadIdx.x; e < vitems; e += blockDim.x) {
    const int dim = e / (len + 1), k = e % (len + 1);
    if (source(k) == k) continue;
    stg(v_cache + base + (size_t)dim * cap + prefix_len + k, vents[e]);
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
