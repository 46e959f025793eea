// Read-only streaming kernels for the benchmark: the measured HBM read
// ceiling that the decode kernel's achieved bandwidth is set beside.  Not
// part of the decode path and not declared in include/art.h; built into
// libart_bench.so, which only bench.py loads.
//
// A workgroup of 256 threads reads four 16 KiB pieces per iteration, each
// thread 16 bytes per 4 KiB of a piece, all sixteen loads issued before any
// is used (64 KiB in flight per workgroup).  Pieces are either consecutive
// (a plain sequential stream over the buffer) or taken from a list of piece
// indices (pages scattered over a pool, as the decode kernel reads a paged
// KV cache).  Every thread folds what it read into one word and writes it
// out, so that no load can be dropped.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kPieceBytes = 16384;
constexpr int kPiecesPerIter = 4;
constexpr int kLoadsPerPiece = kPieceBytes / (kThreads * 16);  // 4

__global__ void __launch_bounds__(kThreads)
read_pieces_kernel(const u32x4* __restrict__ buf, int64_t n_pieces, const int32_t* __restrict__ list,
                   uint32_t* __restrict__ sink) {
  const int tid = threadIdx.x;
  uint32_t acc = 0;
  constexpr int kVecPerPiece = kPieceBytes / 16;
  for (int64_t p0 = (int64_t)blockIdx.x * kPiecesPerIter; p0 < n_pieces;
       p0 += (int64_t)gridDim.x * kPiecesPerIter) {
    u32x4 v[kPiecesPerIter][kLoadsPerPiece];
#pragma unroll
    for (int i = 0; i < kPiecesPerIter; ++i) {
      const int64_t p = p0 + i < n_pieces ? p0 + i : n_pieces - 1;
      const int64_t piece = list ? (int64_t)list[p] : p;
      const u32x4* src = buf + piece * kVecPerPiece + tid;
#pragma unroll
      for (int j = 0; j < kLoadsPerPiece; ++j) v[i][j] = src[j * kThreads];
    }
#pragma unroll
    for (int i = 0; i < kPiecesPerIter; ++i)
#pragma unroll
      for (int j = 0; j < kLoadsPerPiece; ++j) acc ^= v[i][j][0] ^ v[i][j][1] ^ v[i][j][2] ^ v[i][j][3];
  }
  sink[(int64_t)blockIdx.x * kThreads + tid] = acc;
}

}  // namespace

extern "C" {

// Bytes of one piece and threads per workgroup (the caller sizes `sink`:
// grid * 256 words).
int art_bench_piece_bytes(void) { return kPieceBytes; }

// Reads n_pieces pieces of 16 KiB from `buf` (list == NULL: pieces
// 0 .. n_pieces-1 in order; otherwise the pieces list[0 .. n_pieces-1], each
// index < the number of pieces in buf) with `grid` workgroups on `stream`.
// Returns a hipError_t.
int art_bench_read(const void* buf, int64_t n_pieces, const int32_t* list, int32_t grid,
                   uint32_t* sink, hipStream_t stream) {
  if (!buf || !sink || n_pieces <= 0 || grid <= 0) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(read_pieces_kernel, dim3((unsigned)grid), dim3(kThreads), 0, stream,
                     static_cast<const u32x4*>(buf), n_pieces, list, sink);
  return (int)hipGetLastError();
}

}  // extern "C"
