// One-time re-layout of plain W[out][in] matrices into MFMA-fragment order.
//
// Packed image of a matrix with `tiles` 64-column tiles and `ksteps` 32-wide
// k-steps: block (t, s) is 4 KiB at ((t * ksteps + s) * 4 KiB); inside it,
// n-block nb (16 columns) occupies 1 KiB, and lane l's 16 bytes hold
// W[col(64 t + 16 nb + l % 16)][32 s + 8 (l / 16) + e], e = 0..7: exactly the
// B-operand fragment of one 16x16x32 MFMA, so a wave streams its weights with
// one contiguous 1 KiB load per n-block per k-step.  Columns beyond the
// matrix and inputs beyond K are zero.
//
// Column orders:
//  PACK_PLAIN     packed column c is output row c.
//  PACK_QKV_ROPE  each 64-column tile holds 32 dims of one head of q, k or v and
//                 their rotary partners (dim j and j + Dh/2 in the same tile),
//                 so the rotation is applied inside one tile's epilogue.
//  PACK_GATE_UP   tile t holds gate rows [32t, 32t+32) then up rows
//                 [32t, 32t+32), so the SwiGLU product is formed inside one
//                 tile's epilogue; F is padded to a multiple of 32 with zeros.
#include "device.h"
#include "kernels.h"

namespace llmcad {

__device__ __forceinline__ int packed_col_to_row(int c, int N, int kind, int H, int Dh, int F) {
  const int t = c / 64, cc = c % 64;
  if (kind == PACK_PLAIN) return c < N ? c : -1;
  if (kind == PACK_QKV_ROPE) {
    const int tiles_per_head = Dh / 64;
    const int per_part = H * tiles_per_head;
    const int part = t / per_part, r = t % per_part;
    const int h = r / tiles_per_head, b = r % tiles_per_head;
    const int half = Dh / 2;
    const int j = cc < 32 ? 32 * b + cc : half + 32 * b + (cc - 32);
    return part * (H * Dh) + h * Dh + j;
  }
  // PACK_GATE_UP
  const int f = 32 * t + (cc % 32);
  if (f >= F) return -1;
  return cc < 32 ? f : F + f;
}

__global__ void pack_kernel(const bf16* __restrict__ w, int N, int K, bf16x8* __restrict__ out,
                            long total_chunks, int ksteps, int kind, int H, int Dh, int F) {
  for (long ch = blockIdx.x * (long)blockDim.x + threadIdx.x; ch < total_chunks;
       ch += (long)gridDim.x * blockDim.x) {
    const int lane = (int)(ch % 64);
    const long blk = ch / 64;  // (t * ksteps + s) * 4 + nb
    const int nb = (int)(blk % 4);
    const long ts = blk / 4;
    const int s = (int)(ts % ksteps);
    const int t = (int)(ts / ksteps);
    const int c = 64 * t + 16 * nb + lane % 16;
    const int row = packed_col_to_row(c, N, kind, H, Dh, F);
    const int k0 = 32 * s + 8 * (lane / 16);
    bf16x8 v;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int k = k0 + e;
      v[e] = (row >= 0 && k < K) ? w[(long)row * K + k] : (bf16)0.0f;
    }
    out[ch] = v;
  }
}

hipError_t launch_pack(const void* w, int N, int K, void* out, int tiles, int ksteps, int kind,
                       int H, int Dh, int F, hipStream_t st) {
  const long total = (long)tiles * ksteps * 4 * 64;
  long blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  pack_kernel<<<dim3((unsigned)blocks), dim3(256), 0, st>>>((const bf16*)w, N, K, (bf16x8*)out,
                                                             total, ksteps, kind, H, Dh, F);
  return hipGetLastError();
}

}  // namespace llmcad
