// MFMA fragment order of the tensors that one kernel writes and a later one reads as MFMA
// operands (workspace only; the public tensors and debug taps keep their row-major layouts).
//
// An int8 operand of v_mfma_i32_32x32x32_i8 is a 32-row tile with a 32-wide K block; lane l
// holds row l % 32 and the 16 K values starting at 16 (l / 32).  Stored so that the 64 lanes'
// 16-byte slices are consecutive, a wave fetches a whole fragment as one contiguous 1 KB run
// instead of 32 partial rows.
//   kslice order: tile (row / 32, k / 32) at ((row / 32) (K / 32) + k / 32) * 1 KB.
//   permuted kslice order (pk): the same tiles and lane slices, with the K values of a 32-wide
//                 block dealt to the two half-waves in runs of 4: lane l holds, at byte
//                 4 g + i, k = 8 g + 4 (l / 32) + i (g, i < 4).  A contraction is unchanged
//                 when both operands permute K alike, and this is exactly the row order in
//                 which a 32x32 MFMA result leaves its lanes: lane l holds column l % 32 at
//                 rows 8 (r / 4) + 4 (l / 32) + r % 4.  The single-pass scan keeps its chunk
//                 states in this order in registers and hands them on without a transpose.
//   CB order:     the 36 causal 32x32 blocks (J, I <= J) of a 256x256 chunk; lane l of block
//                 (J, I) holds row j = 32 J + l % 32 and the bytes i = 32 I + 16 ks + 8 (l / 32)
//                 + e (ks = 0, 1; e < 8) in the order [ks][e]: the two K-slices of the fp16
//                 32x32x16 ChunkScan2 B operand.  The int8 codes are stored offset by 128
//                 (unsigned byte q + 128; entries i > j hold the code of zero, byte 128),
//                 the form in which ChunkScan2 converts them to fp16.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ssdi8 {
namespace frag {

constexpr int kCbBlocks = 36;
constexpr int kCbChunkBytes = kCbBlocks * 1024;

// Byte offset of element (row, k) of a rows x K int8 matrix (K % 32 == 0) in kslice order;
// consecutive k with the same k / 16 are consecutive bytes.
__host__ __device__ __forceinline__ size_t kslice_offset(int row, int k, int K) {
  const int lane = (row & 31) + 32 * ((k & 31) >> 4);
  return ((size_t)(row >> 5) * (K >> 5) + (k >> 5)) * 1024 + lane * 16 + (k & 15);
}

// Byte offset of element (row, k) in permuted kslice order (see above).
__host__ __device__ __forceinline__ size_t pk_offset(int row, int k, int K) {
  const int kk = k & 31;
  const int lane = (row & 31) + 32 * ((kk >> 2) & 1);
  const int q = 4 * (kk >> 3) + (kk & 3);
  return ((size_t)(row >> 5) * (K >> 5) + (k >> 5)) * 1024 + lane * 16 + q;
}

// Inverse of pk_offset.
__host__ __device__ __forceinline__ void pk_coords(size_t off, int K, int* row, int* k) {
  const size_t blk = off >> 10;
  const int kb = K >> 5;
  const int lane = (int)((off >> 4) & 63);
  const int q = (int)(off & 15);
  *row = (int)(blk / kb) * 32 + (lane & 31);
  *k = (int)(blk % kb) * 32 + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
}

// Inverse of kslice_offset: the (row, k) of byte offset `off`.
__host__ __device__ __forceinline__ void kslice_coords(size_t off, int K, int* row, int* k) {
  const size_t blk = off >> 10;
  const int kb = K >> 5;
  const int lane = (int)((off >> 4) & 63);
  *row = (int)(blk / kb) * 32 + (lane & 31);
  *k = (int)(blk % kb) * 32 + 16 * (lane >> 5) + (int)(off & 15);
}

// Index of causal block (J, I), I <= J, within a chunk.
__host__ __device__ __forceinline__ int cb_block(int J, int I) { return J * (J + 1) / 2 + I; }

// Byte offset of in-block element (jj, ii) (0 <= jj, ii < 32) within its 1 KB CB block.
__host__ __device__ __forceinline__ int cb_inblock(int jj, int ii) {
  return (jj + 32 * ((ii >> 3) & 1)) * 16 + (ii >> 4) * 8 + (ii & 7);
}

// fp16 operands of v_mfma_f32_32x32x16_f16 (and the fp32 states they are converted from): a
// 32-row x 16-K tile of 512 elements, lane l holding row l % 32 and the 8 K values starting at
// 8 (l / 32).  Element offset of (row, k) of a rows x K matrix (K % 16 == 0).
__host__ __device__ __forceinline__ size_t k16_offset(int row, int k, int K) {
  const int lane = (row & 31) + 32 * ((k & 15) >> 3);
  return ((size_t)(row >> 5) * (K >> 4) + (k >> 4)) * 512 + lane * 8 + (k & 7);
}

// Inverse of k16_offset.
__host__ __device__ __forceinline__ void k16_coords(size_t off, int K, int* row, int* k) {
  const size_t tile = off >> 9;
  const int kt = K >> 4;
  const int lane = (int)((off >> 3) & 63);
  *row = (int)(tile / kt) * 32 + (lane & 31);
  *k = (int)(tile % kt) * 16 + 8 * (lane >> 5) + (int)(off & 7);
}

}  // namespace frag
}  // namespace ssdi8
