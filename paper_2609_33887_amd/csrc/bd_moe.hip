// Mixture-of-experts FFN pieces: router (softmax, top-k, renormalised
// weights), deterministic expert dispatch, and the fixed-order combine.  The
// expert products themselves run in the grouped MFMA GEMM (bd_gemm.hip).
#include "bd_internal.h"

#include <math.h>

namespace bd {

__device__ __forceinline__ float bf2f_e(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// Router.  A workgroup takes 16 rows with 16 waves: wave (q, w) multiplies
// depth quarter q of the logits of experts 16 w .. 16 w + 15 on the fp32
// matrix cores (v_mfma_f32_16x16x4_f32: fp32 operands, fp32 accumulation):
// the A operand is the row's activation pair summed in fp32 (hi + lo), the
// B operand the fp32 router weights [E][d] read straight from global memory
// (one 64-byte run per lane and block; the next block's loads are in flight
// while the current one is multiplied, and the workgroup's 16 waves cover
// each other's load latency).  In MFMA step s of the 64-deep block at k0, lane group g feeds
// depth k0 + 16 g + s; four accumulators take the steps s mod 4; the four
// quarters are summed in LDS in a fixed order (an fp32 sum of the same
// products in another order than the plain dot product).  Then one wave per
// row: softmax over the E lanes, top_k selection by repeated wave argmax
// (lowest expert id among equal probabilities), and weights renormalised
// over the chosen experts.  Needs E <= 64 and d % 256 == 0.
constexpr int RR = 16;     // rows per workgroup (one per wave in the tail)
constexpr int RKB = 64;    // depth per block
constexpr int RQ = 4;      // depth quarters
__global__ __launch_bounds__(1024) void k_router(const bf16_t* __restrict__ A, size_t a_plane, int d,
                                                 const float* __restrict__ Wr, int E, int topk,
                                                 const int32_t* __restrict__ Mp,
                                                 int32_t* __restrict__ top_e, float* __restrict__ top_w) {
  __shared__ float sP[RQ][RR][65];
  const int M = *Mp;
  const int row0 = blockIdx.x * RR;
  if (row0 >= M) return;
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const int wq = wave >> 2, we = wave & 3;
  const int g = lane >> 4, c = lane & 15;
  const bool rv = row0 + c < M;               // this lane's A row is live
  const int e = we * 16 + c;
  const bool ev = e < E;                      // this lane's expert exists
  const int kq = d / RQ, kbeg = wq * kq;
  const bf16_t* ap = A + (size_t)(rv ? row0 + c : row0) * d + kbeg + 16 * g;
  const float* wp = Wr + (size_t)(ev ? e : 0) * d + kbeg + 16 * g;
  u32x4 ah[2], al[2];
  float4 wv[4];
  auto fetch = [&](int k0) {
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      ah[x] = *(const u32x4*)(ap + k0 + 8 * x);
      al[x] = *(const u32x4*)(ap + k0 + 8 * x + a_plane);
    }
#pragma unroll
    for (int x = 0; x < 4; ++x) wv[x] = *(const float4*)(wp + k0 + 4 * x);
  };
  floatx4 acc[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) acc[q] = floatx4{0.f, 0.f, 0.f, 0.f};
  fetch(0);
  for (int k0 = 0; k0 < kq; k0 += RKB) {
    float a[16], w[16];
    const bf16_t* h = (const bf16_t*)ah;
    const bf16_t* l = (const bf16_t*)al;
#pragma unroll
    for (int x = 0; x < 16; ++x) a[x] = rv ? bf2f_e(h[x]) + bf2f_e(l[x]) : 0.f;
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      w[4 * x] = ev ? wv[x].x : 0.f;
      w[4 * x + 1] = ev ? wv[x].y : 0.f;
      w[4 * x + 2] = ev ? wv[x].z : 0.f;
      w[4 * x + 3] = ev ? wv[x].w : 0.f;
    }
    if (k0 + RKB < kq) fetch(k0 + RKB);
#pragma unroll
    for (int s2 = 0; s2 < 16; ++s2)
      acc[s2 & 3] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s2], w[s2], acc[s2 & 3], 0, 0, 0);
  }
  // lane (g, c) holds quarter wq of the logits of rows 4 g + i, expert e
#pragma unroll
  for (int i = 0; i < 4; ++i) sP[wq][4 * g + i][e] = (acc[0][i] + acc[1][i]) + (acc[2][i] + acc[3][i]);
  __syncthreads();
  {
    const int rr = wave;
    const int row = row0 + rr;
    if (row >= M) return;
    const float lg = (sP[0][rr][lane] + sP[1][rr][lane]) + (sP[2][rr][lane] + sP[3][rr][lane]);
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

hipError_t launch_router(const void* A, size_t a_plane, int d, const float* Wr, int E, int topk,
                         const int32_t* M_dev, int rows_cap, int32_t* top_e, float* top_w,
                         hipStream_t st) {
  if (E > 64 || topk > E || topk < 1 || d % (RQ * RKB)) return hipErrorInvalidValue;
  k_router<<<(rows_cap + RR - 1) / RR, 1024, 0, st>>>((const bf16_t*)A, a_plane, d, Wr, E, topk, M_dev,
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

}  // namespace bd
