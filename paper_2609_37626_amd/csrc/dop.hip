// gfx950 kernels of the DOP regroup around the attention step (Sec. 3 "DOP:
// Computation"; App. E, DOP transfer).  With sharded projections, rank t
// holds all N current query rows for its H_l = H/T heads; the owner of a
// request needs that request's rows for all H heads.  A variable all-to-all
// moves the blocks between them (not part of this library); these kernels
// build and take apart the blocks on either side:
//   pack_q    rank:  send[k][h]        = q_nope[order[k]][h] | q_rope[order[k]][h]
//   unpack_q  owner: q_owner[i][tH_l+h] = recv[t][i][h]
//   pack_out  owner: send[t][i][h]     = out_owner[i][tH_l+h]
//   unpack_out rank: out[order[k]][h]  = recv[k][h]
// order lists the rows grouped by owner, so the send and receive buffers
// hold one contiguous block per peer.  Rows keep their identity, heads their
// order, and the no-position and rotary query parts travel in one row.
// Pure data movement: one wave per row, one 16-byte piece per lane (a bf16
// row of 576 is 72 pieces, of 512 is 64).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.hpp"

namespace splash {

namespace {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kQPieces = 72;    // 576 bf16
constexpr int kNopePieces = 64;  // 512 bf16
constexpr int kRopePieces = 8;   // 64 bf16
constexpr int kOutPieces = 64;   // 512 bf16

__device__ __forceinline__ int32_t wave_id() { return (int32_t)((blockIdx.x * blockDim.x + threadIdx.x) >> 6); }
__device__ __forceinline__ int32_t num_waves() { return (int32_t)((gridDim.x * blockDim.x) >> 6); }

__global__ __launch_bounds__(256) void dop_pack_q_kernel(const u32x4* __restrict__ nope,
                                                         const u32x4* __restrict__ rope,
                                                         const int32_t* __restrict__ order, int32_t n, int32_t hl,
                                                         u32x4* __restrict__ send) {
  const int lane = threadIdx.x & 63;
  for (int32_t r = wave_id(); r < n * hl; r += num_waves()) {  // send row r = k * hl + h
    const int32_t k = r / hl, h = r - k * hl;
    const int64_t src = (int64_t)order[k] * hl + h;
    u32x4* dst = send + (int64_t)r * kQPieces;
    dst[lane] = nope[src * kNopePieces + lane];
    if (lane < kRopePieces) dst[kNopePieces + lane] = rope[src * kRopePieces + lane];
  }
}

__global__ __launch_bounds__(256) void dop_unpack_q_kernel(const u32x4* __restrict__ recv, int32_t T, int32_t n,
                                                           int32_t hl, u32x4* __restrict__ q_owner) {
  const int lane = threadIdx.x & 63;
  const int32_t H = T * hl;
  for (int32_t r = wave_id(); r < n * H; r += num_waves()) {  // owner row r = i * H + hh
    const int32_t i = r / H, hh = r - i * H, t = hh / hl, h = hh - t * hl;
    const u32x4* src = recv + ((int64_t)(t * n + i) * hl + h) * kQPieces;
    u32x4* dst = q_owner + (int64_t)r * kQPieces;
    dst[lane] = src[lane];
    if (lane < kQPieces - 64) dst[64 + lane] = src[64 + lane];
  }
}

__global__ __launch_bounds__(256) void dop_pack_out_kernel(const u32x4* __restrict__ out_owner, int32_t T, int32_t n,
                                                           int32_t hl, u32x4* __restrict__ send) {
  const int lane = threadIdx.x & 63;
  const int32_t H = T * hl, per_rank = n * hl;
  for (int32_t r = wave_id(); r < T * per_rank; r += num_waves()) {  // send row r = (t * n + i) * hl + h
    const int32_t t = r / per_rank, rem = r - t * per_rank, i = rem / hl, h = rem - i * hl;
    send[(int64_t)r * kOutPieces + lane] = out_owner[((int64_t)i * H + t * hl + h) * kOutPieces + lane];
  }
}

__global__ __launch_bounds__(256) void dop_unpack_out_kernel(const u32x4* __restrict__ recv,
                                                             const int32_t* __restrict__ order, int32_t n, int32_t hl,
                                                             u32x4* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  for (int32_t r = wave_id(); r < n * hl; r += num_waves()) {  // receive row r = k * hl + h
    const int32_t k = r / hl, h = r - k * hl;
    out[((int64_t)order[k] * hl + h) * kOutPieces + lane] = recv[(int64_t)r * kOutPieces + lane];
  }
}

unsigned grid_for(int64_t rows) {
  int64_t blocks = (rows + 3) / 4;  // four waves (rows) per block and pass
  if (blocks > 8192) blocks = 8192;
  return (unsigned)(blocks < 1 ? 1 : blocks);
}

}  // namespace

hipError_t launch_dop_pack_q(const void* q_nope, const void* q_rope, const int32_t* order, int32_t n, int32_t hl,
                             void* send, hipStream_t s) {
  hipLaunchKernelGGL(dop_pack_q_kernel, dim3(grid_for((int64_t)n * hl)), dim3(256), 0, s, (const u32x4*)q_nope,
                     (const u32x4*)q_rope, order, n, hl, (u32x4*)send);
  return hipGetLastError();
}

hipError_t launch_dop_unpack_q(const void* recv, int32_t T, int32_t n, int32_t hl, void* q_owner, hipStream_t s) {
  hipLaunchKernelGGL(dop_unpack_q_kernel, dim3(grid_for((int64_t)n * T * hl)), dim3(256), 0, s, (const u32x4*)recv,
                     T, n, hl, (u32x4*)q_owner);
  return hipGetLastError();
}

hipError_t launch_dop_pack_out(const void* out_owner, int32_t T, int32_t n, int32_t hl, void* send, hipStream_t s) {
  hipLaunchKernelGGL(dop_pack_out_kernel, dim3(grid_for((int64_t)n * T * hl)), dim3(256), 0, s,
                     (const u32x4*)out_owner, T, n, hl, (u32x4*)send);
  return hipGetLastError();
}

hipError_t launch_dop_unpack_out(const void* recv, const int32_t* order, int32_t n, int32_t hl, void* out,
                                 hipStream_t s) {
  hipLaunchKernelGGL(dop_unpack_out_kernel, dim3(grid_for((int64_t)n * hl)), dim3(256), 0, s, (const u32x4*)recv,
                     order, n, hl, (u32x4*)out);
  return hipGetLastError();
}

}  // namespace splash
