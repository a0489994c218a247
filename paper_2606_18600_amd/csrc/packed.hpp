// Fragment-packed bf16 layouts read by the MFMA GEMMs.
//
// Both layouts store whole v_mfma_f32_16x16x32_bf16 operand fragments
// contiguously: a fragment is 16 rows x 32 k, 1 KB, held lane-major, lane l
// owning row (l % 16) and k offsets (l / 16) * 8 .. + 7 (16 bytes). A wave
// therefore loads a fragment with one fully contiguous 1 KB access.
//
// Activations (the A operand, [M, K], M padded to a multiple of 16):
//   fragment (m / 16, k / 32) at index (m / 16) * (K / 32) + k / 32.
// Weights (the B operand, [N, K], N % 64 == 0): rows are grouped by 64; a
// group's fragments for one k step are adjacent, so streaming a group over K
// reads one contiguous range:
//   fragment index ((n / 64) * (K / 32) + k / 32) * 4 + (n / 16) % 4.
// For the fused gate-up weight, packed row 64 g + r holds gate row 32 g + r
// for r < 32 and up row 32 g + r - 32 otherwise, so every 64-row group
// produces the gate and up halves of the same 32 SwiGLU outputs.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace stage_k {

__host__ __device__ inline size_t packed_a_offset(int m, int k, int K) {
  const size_t frag = (size_t)(m >> 4) * (K >> 5) + (k >> 5);
  const int lane = (m & 15) + 16 * ((k & 31) >> 3);
  return frag * 512 + lane * 8 + (k & 7);
}

__host__ __device__ inline size_t packed_w_offset(int n, int k, int K) {
  const size_t frag = ((size_t)(n >> 6) * (K >> 5) + (k >> 5)) * 4 + ((n >> 4) & 3);
  const int lane = (n & 15) + 16 * ((k & 31) >> 3);
  return frag * 512 + lane * 8 + (k & 7);
}

// Row of the unpacked gate-up matrix [gate (F rows); up (F rows)] stored at
// packed row n.
__host__ __device__ inline int gate_up_source_row(int n, int F) {
  const int g = n >> 6, r = n & 63;
  return r < 32 ? 32 * g + r : F + 32 * g + (r - 32);
}

// KV cache: per (layer, block, kv head) a K plane and a V plane of
// block_size (16) tokens x d, each stored as whole MFMA operand fragments.
// K plane: fragments of 16 tokens x 32 d (the A operand of S^T = K Q^T);
// lane l holds token l % 16, d offsets (l / 16) * 8 .. + 7 of the fragment.
__host__ __device__ inline int kv_k_offset(int o, int d) {
  return (d >> 5) * 512 + (o + 16 * ((d & 31) >> 3)) * 8 + (d & 7);
}
// V plane: the A operands of O^T += V^T P^T are 16 d x 16 tokens (lane l:
// d = l % 16, tokens (l / 16) * 4 .. + 3, 8 bytes); two d tiles 2p, 2p + 1
// are interleaved per lane so that one 16-byte load per lane (a 1 KB
// fragment) fetches both: lane l holds tile 2p's 4 tokens, then tile 2p+1's.
__host__ __device__ inline int kv_v_offset(int o, int d) {
  return (d >> 5) * 512 + ((d & 15) + 16 * (o >> 2)) * 8 + ((d >> 4) & 1) * 4 + (o & 3);
}

}  // namespace stage_k
