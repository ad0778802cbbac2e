// Mixture-of-experts FFN pieces: router (softmax, top-k, renormalised
// weights), deterministic expert dispatch, and the fixed-order combine.  The
// expert products themselves run in the grouped MFMA GEMM (bd_gemm.hip).
#include "bd_internal.h"

#include <math.h>

namespace bd {

__device__ __forceinline__ float bf2f_e(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// Router.  A workgroup takes 16 rows: thread t accumulates the logits of
// experts 4 (t % 16) + [0, 4) of row t / 16 over d in chunks of RC = 128,
// the row's activation pair (hi + lo, summed in fp32) and the transposed fp32
// router weights staged in LDS (the weights are read once per workgroup, not
// once per row; the next chunk's loads are in flight, in registers, while
// the current chunk is computed); every logit is the FMA chain over
// k = 0 .. d-1 in order.  Then one wave per row: softmax over the E lanes,
// top_k selection by repeated wave argmax (lowest expert id among equal
// probabilities), and weights renormalised over the chosen experts.
// Needs E <= 64 and d % 128 == 0.
constexpr int RR = 16;     // rows per workgroup
constexpr int RC = 128;    // k per LDS chunk
__global__ __launch_bounds__(256) void k_router(const bf16_t* __restrict__ A, size_t a_plane, int d,
                                                const float* __restrict__ WrT, int E, int topk,
                                                const int32_t* __restrict__ Mp,
                                                int32_t* __restrict__ top_e, float* __restrict__ top_w) {
  __shared__ float sA[RR][RC + 4];
  __shared__ __attribute__((aligned(16))) float sW[RC][64];
  __shared__ float sL[RR][65];
  const int M = *Mp;
  const int row0 = blockIdx.x * RR;
  if (row0 >= M) return;
  const int t = threadIdx.x;
  const int r = t / 16, e0 = (t % 16) * 4;
  // staging assignment: A -- row t / 16, k = 8 (t % 16) + [0, 8) (one 16-byte
  // load per plane); W -- float4 i of the chunk's RC x 64 block for
  // i = t + 256 j, j < 8 (k = i / 16, experts 4 (i % 16) + [0, 4))
  const int ar = t / 16, ak = (t % 16) * 8;
  const bool arow = row0 + ar < M;
  const bf16_t* ap = A + (size_t)(arow ? row0 + ar : row0) * d + ak;
  u32x4 ah, al;
  float4 wv[8];
  auto fetch = [&](int k0) {
    ah = *(const u32x4*)(ap + k0);
    al = *(const u32x4*)(ap + k0 + a_plane);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int i = t + 256 * j, kk = i / 16, e = (i % 16) * 4;
      if (E == 64) {
        wv[j] = *(const float4*)(WrT + (size_t)(k0 + kk) * 64 + e);
      } else {
        float v[4];
#pragma unroll
        for (int x = 0; x < 4; ++x) v[x] = e + x < E ? WrT[(size_t)(k0 + kk) * E + e + x] : 0.f;
        wv[j] = make_float4(v[0], v[1], v[2], v[3]);
      }
    }
  };
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  fetch(0);
  for (int k0 = 0; k0 < d; k0 += RC) {
    const bf16_t* h = (const bf16_t*)&ah;
    const bf16_t* l = (const bf16_t*)&al;
#pragma unroll
    for (int x = 0; x < 8; ++x) sA[ar][ak + x] = arow ? bf2f_e(h[x]) + bf2f_e(l[x]) : 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int i = t + 256 * j;
      *(float4*)&sW[i / 16][(i % 16) * 4] = wv[j];
    }
    __syncthreads();
    if (k0 + RC < d) fetch(k0 + RC);
#pragma unroll 8
    for (int kk = 0; kk < RC; ++kk) {
      const float a = sA[r][kk];
      const float4 w = *(const float4*)&sW[kk][e0];
      acc[0] = fmaf(a, w.x, acc[0]);
      acc[1] = fmaf(a, w.y, acc[1]);
      acc[2] = fmaf(a, w.z, acc[2]);
      acc[3] = fmaf(a, w.w, acc[3]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) sL[r][e0 + j] = acc[j];
  __syncthreads();
  const int wave = t >> 6, lane = t & 63;
  for (int rr = wave; rr < RR; rr += 4) {
    const int row = row0 + rr;
    if (row >= M) break;
    const float lg = sL[rr][lane];
    float mx = lane < E ? lg : -INFINITY;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    const float p = lane < E ? expf(lg - mx) : 0.f;
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
}

hipError_t launch_router(const void* A, size_t a_plane, int d, const float* WrT, int E, int topk,
                         const int32_t* M_dev, int rows_cap, int32_t* top_e, float* top_w,
                         hipStream_t st) {
  if (E > 64 || topk > E || topk < 1 || d % RC) return hipErrorInvalidValue;
  k_router<<<(rows_cap + RR - 1) / RR, 256, 0, st>>>((const bf16_t*)A, a_plane, d, WrT, E, topk, M_dev,
                                                     top_e, top_w);
  return hipGetLastError();
}

// Dispatch: one workgroup per expert.  Every workgroup first histograms all
// assignments by expert in LDS (integer atomics: exact counts), which gives
// its expert's offset in the expert-sorted order and its tiles; then it
// visits the assignments in (row, slot) order with wave ballots and prefix
// counts, so each expert's list is sorted by token row.
__global__ __launch_bounds__(256) void k_moe_scatter(const int32_t* __restrict__ top_e, int topk, int E,
                                                     const int32_t* __restrict__ Mp, MoeLists L) {
  __shared__ int hist[64];
  __shared__ int wtot[4];
  const int e = blockIdx.x;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int n = *Mp * topk;
  if (threadIdx.x < 64) hist[threadIdx.x] = 0;
  __syncthreads();
  for (int i = threadIdx.x; i < n; i += blockDim.x) atomicAdd(&hist[top_e[i]], 1);
  __syncthreads();
  int off = 0, toff = 0, total_tiles = 0;
  for (int k = 0; k < E; ++k) {
    const int c = hist[k];
    const int nt = (c + GROUP_BM - 1) / GROUP_BM;
    if (k < e) { off += c; toff += nt; }
    total_tiles += nt;
  }
  const int cnt = hist[e];
  if (threadIdx.x == 0) {
    L.e_cnt[e] = cnt;
    L.e_off[e] = off;
    if (e == 0) L.ntiles[0] = total_tiles;
  }
  for (int t = threadIdx.x; t * GROUP_BM < cnt; t += blockDim.x) {
    L.tile_e[toff + t] = e;
    L.tile_m0[toff + t] = t * GROUP_BM;
  }
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
  if (E > 64) return hipErrorInvalidValue;
  k_moe_scatter<<<E, 256, 0, st>>>(top_e, topk, E, M_dev, L);
  return hipGetLastError();
}

// X[row] += sum_j w_j Y[pos_j] over the row's top_k slots in rank order
// (fixed order); each thread 4 consecutive columns.
__global__ __launch_bounds__(256) void k_moe_combine(float* __restrict__ X, const float* __restrict__ Y,
                                                     const int32_t* __restrict__ pos_of,
                                                     const float* __restrict__ top_w, int topk, int d,
                                                     const int32_t* __restrict__ Mp) {
  const int row = blockIdx.y;
  if (row >= *Mp) return;
  const int c = (blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (c >= d) return;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int j = 0; j < topk; ++j) {
    const size_t k = (size_t)row * topk + j;
    const float w = top_w[k];
    const float4 y = *(const float4*)(Y + (size_t)pos_of[k] * d + c);
    acc.x += w * y.x; acc.y += w * y.y; acc.z += w * y.z; acc.w += w * y.w;
  }
  float4* x = (float4*)(X + (size_t)row * d + c);
  float4 v = *x;
  v.x += acc.x; v.y += acc.y; v.z += acc.z; v.w += acc.w;
  *x = v;
}

hipError_t launch_moe_combine(float* X, const float* Y, const int32_t* pos_of, const float* top_w,
                              int topk, int d, const int32_t* M_dev, int rows_cap, hipStream_t st) {
  if (d % 4) return hipErrorInvalidValue;
  k_moe_combine<<<dim3((d / 4 + 255) / 256, rows_cap), 256, 0, st>>>(X, Y, pos_of, top_w, topk, d, M_dev);
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
