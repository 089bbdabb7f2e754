// One-time re-layout of plain W[out][in] matrices into MFMA-fragment order.
//
// Packed image of a matrix with `nblocks` 16-column blocks and `ksteps`
// 32-wide k-steps: block-major, block (nb, s) is 1 KiB at
// ((nb * ksteps + s) * 1 KiB), and lane l's 16 bytes hold
// W[col(16 nb + l % 16)][32 s + 8 (l / 16) + e], e = 0..7 -- exactly the B
// operand of one 16x16x32 MFMA.  A wave streams a block's weights with one
// contiguous 1 KiB load per k-step, and consecutive k-steps are consecutive
// KiBs.  Columns beyond the matrix and inputs beyond K are zero.
//
// Column orders:
//  PACK_PLAIN     packed column c is output row c.
//  PACK_GATE_UP   block i holds gate rows [8i, 8i+8) then up rows [8i, 8i+8),
//                 so the SwiGLU product of 8 columns is formed inside one
//                 block; F is padded to a multiple of 32 with zeros.
//  PACK_QKV_ROPE  the fused [q; k; v] projection (N = 3d rows).  In the q and
//                 k parts, block t of a head (Dh / 16 per head) holds that
//                 head's dims [8t, 8t+8) then [8t + Dh/2, 8t + Dh/2 + 8): the
//                 pairs the rotary embedding mixes (rotate-half pairing, dim j
//                 with j + Dh/2) sit 8 columns apart inside one block.  The v
//                 part is plain.
#include "device.h"
#include "kernels.h"
#include "layout.h"

namespace llmcad {

__device__ __forceinline__ int packed_col_to_row(int c, int N, int kind, int aux) {
  if (kind == PACK_PLAIN) return c < N ? c : -1;
  if (kind == PACK_QKV_ROPE) {
    const int d = N / 3, dh = aux;
    if (c >= 2 * d) return c < N ? c : -1;
    const int part = c / d, cq = c % d, head = cq / dh, w = cq % dh;
    const int t = w / kNB, ci = w % kNB;
    return part * d + head * dh + 8 * t + (ci % 8) + (ci < 8 ? 0 : dh / 2);
  }
  const int F = aux;
  const int nb = c / kNB, cc = c % kNB;
  const int f = 8 * nb + (cc % 8);
  if (f >= F) return -1;
  return cc < 8 ? f : F + f;
}

__global__ void pack_kernel(const bf16* __restrict__ w, int N, int K, bf16x8* __restrict__ out,
                            long total_chunks, int ksteps, int kind, int aux) {
  for (long ch = blockIdx.x * (long)blockDim.x + threadIdx.x; ch < total_chunks;
       ch += (long)gridDim.x * blockDim.x) {
    const int lane = (int)(ch % 64);
    const long blk = ch / 64;  // nb * ksteps + s
    const int s = (int)(blk % ksteps);
    const int nb = (int)(blk / ksteps);
    const int row = packed_col_to_row(kNB * nb + lane % 16, N, kind, aux);
    const int k0 = kStepK * s + 8 * (lane / 16);
    bf16x8 v;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int k = k0 + e;
      v[e] = (row >= 0 && k < K) ? w[(long)row * K + k] : (bf16)0.0f;
    }
    out[ch] = v;
  }
}

// 4-bit matrices.  Packed codes: block-major, (block nb, group g) is 1 KiB
// at ((nb * groups + g) KiB); lane l's 16 bytes hold column col(16 nb + l % 16)
// for the group's four 32-input k-steps t, one dword each, inputs
// 128 g + 32 t + 8 (l / 16) + e, e = 0..7: code e = 2 p sits in bits
// [4 p, 4 p + 4), code e = 2 p + 1 in bits [16 + 4 p, 20 + 4 p), so that
// (dword >> 4 p) & 0x000F000F, ORed with the bf16 pattern of 128, is the pair
// (128 + q_2p, 128 + q_2p+1) as two bf16 values.  Packed scales: (nb, g) holds
// 16 bf16, column order as the codes.  Absent columns get code 8 and scale 0.
__global__ void pack_q4_kernel(const uint8_t* __restrict__ codes, const bf16* __restrict__ scales, int N, int K,
                               uint32_t* __restrict__ out_codes, bf16* __restrict__ out_scales, long total_lanes,
                               int groups, int kind, int aux) {
  for (long ch = blockIdx.x * (long)blockDim.x + threadIdx.x; ch < total_lanes;
       ch += (long)gridDim.x * blockDim.x) {
    const int lane = (int)(ch % 64);
    const long blk = ch / 64;  // nb * groups + g
    const int g = (int)(blk % groups);
    const int nb = (int)(blk / groups);
    const int row = packed_col_to_row(kNB * nb + lane % 16, N, kind, aux);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      uint32_t word = 0;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int k = kQ4Group * g + kStepK * t + 8 * (lane / 16) + e;
        uint32_t q = 8;
        if (row >= 0 && k < K) q = (codes[(long)row * (K / 2) + k / 2] >> (4 * (k & 1))) & 0xF;
        word |= q << ((e & 1) ? 16 + 4 * (e / 2) : 4 * (e / 2));
      }
      out_codes[ch * 4 + t] = word;
    }
    if (lane < kNB) out_scales[blk * kNB + lane] = row >= 0 ? scales[(long)row * (K / kQ4Group) + g] : (bf16)0.0f;
  }
}

hipError_t launch_pack_q4(const void* codes, const void* scales, int N, int K, void* out_codes, void* out_scales,
                          int nblocks, int groups, int kind, int aux, hipStream_t st) {
  const long total = (long)nblocks * groups * 64;
  long blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  pack_q4_kernel<<<dim3((unsigned)blocks), dim3(256), 0, st>>>((const uint8_t*)codes, (const bf16*)scales, N, K,
                                                                (uint32_t*)out_codes, (bf16*)out_scales, total,
                                                                groups, kind, aux);
  return hipGetLastError();
}

hipError_t launch_pack(const void* w, int N, int K, void* out, int nblocks, int ksteps, int kind,
                       int aux, hipStream_t st) {
  const long total = (long)nblocks * ksteps * 64;
  long blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  pack_kernel<<<dim3((unsigned)blocks), dim3(256), 0, st>>>((const bf16*)w, N, K, (bf16x8*)out,
                                                             total, ksteps, kind, aux);
  return hipGetLastError();
}

}  // namespace llmcad
