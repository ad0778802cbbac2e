// Mixture-of-experts FFN pieces: router (softmax, top-k, renormalised
// weights), deterministic expert dispatch, and the fixed-order combine.  The
// expert products themselves run in the grouped MFMA GEMM (bd_gemm.hip).
#include "bd_internal.h"

#include <math.h>

namespace bd {

__device__ __forceinline__ float bf2f_e(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// One wave per row; lane e computes router logit e = a . Wr[e] from the
// row's activation pair (hi + lo) staged in LDS and the transposed router
// weights (coalesced across lanes).  Then softmax over the E lanes, top_k
// selection by repeated wave argmax (lowest expert id among equal
// probabilities), and weights renormalised over the chosen experts.
__global__ __launch_bounds__(256) void k_router(const bf16_t* __restrict__ A, size_t a_plane, int d,
                                                const float* __restrict__ WrT, int E, int topk,
                                                const int32_t* __restrict__ Mp,
                                                int32_t* __restrict__ top_e, float* __restrict__ top_w) {
  extern __shared__ float sa[];             // [4][d]
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + wave;
  const bool active = row < *Mp;
  float* my = sa + (size_t)wave * d;
  if (active)
    for (int c = lane; c < d; c += 64)
      my[c] = bf2f_e(A[(size_t)row * d + c]) + bf2f_e(A[(size_t)row * d + c + a_plane]);
  __syncthreads();
  if (!active) return;
  float acc = 0.f;
  if (lane < E) {
#pragma unroll 8
    for (int k = 0; k < d; ++k) acc += my[k] * WrT[(size_t)k * E + lane];
  }
  float mx = lane < E ? acc : -INFINITY;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  const float p = lane < E ? expf(acc - mx) : 0.f;
  float ssum = p;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ssum += __shfl_xor(ssum, off);
  float prob = lane < E ? p / ssum : -1.f;
  float chosen_sum = 0.f, my_w = 0.f;
  int my_rank = -1;
  for (int j = 0; j < topk; ++j) {
    float bv = prob;
    int bi = lane;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const float ov = __shfl_xor(bv, off);
      const int oi = __shfl_xor(bi, off);
      if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
    }
    chosen_sum += bv;
    if (lane == bi) { my_rank = j; my_w = prob; prob = -1.f; }
  }
  if (my_rank >= 0) {
    top_e[(size_t)row * topk + my_rank] = lane;
    top_w[(size_t)row * topk + my_rank] = my_w / chosen_sum;
  }
}

hipError_t launch_router(const void* A, size_t a_plane, int d, const float* WrT, int E, int topk,
                         const int32_t* M_dev, int rows_cap, int32_t* top_e, float* top_w,
                         hipStream_t st) {
  if (E > 64 || topk > E || topk < 1) return hipErrorInvalidValue;
  k_router<<<(rows_cap + 3) / 4, 256, 4 * (size_t)d * sizeof(float), st>>>(
      (const bf16_t*)A, a_plane, d, WrT, E, topk, M_dev, top_e, top_w);
  return hipGetLastError();
}

// Counting pass: one workgroup per expert counts its assignments.
__global__ __launch_bounds__(256) void k_moe_count(const int32_t* __restrict__ top_e, int topk,
                                                   const int32_t* __restrict__ Mp,
                                                   int32_t* __restrict__ e_cnt) {
  __shared__ int part[4];
  const int e = blockIdx.x;
  const int n = *Mp * topk;
  int c = 0;
  for (int i = threadIdx.x; i < n; i += blockDim.x) c += (top_e[i] == e);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) e_cnt[e] = part[0] + part[1] + part[2] + part[3];
}

// Scatter pass: one workgroup per expert; assignments are visited in
// (row, slot) order, so each expert's list is sorted by token row.
__global__ __launch_bounds__(256) void k_moe_scatter(const int32_t* __restrict__ top_e, int topk, int E,
                                                     const int32_t* __restrict__ Mp, MoeLists L) {
  __shared__ int wtot[4];
  const int e = blockIdx.x;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int off = 0, toff = 0, total_tiles = 0;
  for (int k = 0; k < E; ++k) {
    const int c = L.e_cnt[k];
    const int nt = (c + GROUP_BM - 1) / GROUP_BM;
    if (k < e) { off += c; toff += nt; }
    total_tiles += nt;
  }
  const int cnt = L.e_cnt[e];
  if (threadIdx.x == 0) {
    L.e_off[e] = off;
    if (e == 0) L.ntiles[0] = total_tiles;
  }
  for (int t = threadIdx.x; t * GROUP_BM < cnt; t += blockDim.x) {
    L.tile_e[toff + t] = e;
    L.tile_m0[toff + t] = t * GROUP_BM;
  }
  const int n = *Mp * topk;
  int run = 0;
  for (int base = 0; base < n; base += blockDim.x) {
    const int i = base + threadIdx.x;
    const bool match = i < n && top_e[i] == e;
    const unsigned long long bal = __ballot(match);
    const int pre = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) wtot[wave] = __popcll(bal);
    __syncthreads();
    int wpre = 0;
    for (int w = 0; w < wave; ++w) wpre += wtot[w];
    if (match) {
      const int pos = off + run + wpre + pre;
      L.list_row[pos] = i / topk;
      L.pos_of[i] = pos;
    }
    run += wtot[0] + wtot[1] + wtot[2] + wtot[3];
    __syncthreads();
  }
}

hipError_t launch_moe_dispatch(const int32_t* top_e, int topk, int E, const int32_t* M_dev,
                               const MoeLists& L, hipStream_t st) {
  k_moe_count<<<E, 256, 0, st>>>(top_e, topk, M_dev, L.e_cnt);
  k_moe_scatter<<<E, 256, 0, st>>>(top_e, topk, E, M_dev, L);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void k_moe_combine(float* __restrict__ X, const float* __restrict__ Y,
                                                     const int32_t* __restrict__ pos_of,
                                                     const float* __restrict__ top_w, int topk, int d,
                                                     const int32_t* __restrict__ Mp) {
  const int row = blockIdx.y;
  if (row >= *Mp) return;
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= d) return;
  float acc = 0.f;
  for (int j = 0; j < topk; ++j) {
    const size_t k = (size_t)row * topk + j;
    acc += top_w[k] * Y[(size_t)pos_of[k] * d + c];
  }
  X[(size_t)row * d + c] += acc;
}

hipError_t launch_moe_combine(float* X, const float* Y, const int32_t* pos_of, const float* top_w,
                              int topk, int d, const int32_t* M_dev, int rows_cap, hipStream_t st) {
  k_moe_combine<<<dim3((d + 255) / 256, rows_cap), 256, 0, st>>>(X, Y, pos_of, top_w, topk, d, M_dev);
  return hipGetLastError();
}

__global__ void k_transpose_f32(const float* __restrict__ in, float* __restrict__ out, int rows,
                                int cols) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (size_t)rows * cols) return;
  const int r = (int)(i / cols), c = (int)(i % cols);
  out[(size_t)c * rows + r] = in[i];
}

hipError_t launch_transpose_f32(const float* in, float* out, int rows, int cols, hipStream_t st) {
  const size_t n = (size_t)rows * cols;
  k_transpose_f32<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(in, out, rows, cols);
  return hipGetLastError();
}

}  // namespace bd
