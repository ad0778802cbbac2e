// Projection GEMMs and the fused LM-head softmax-statistics kernel.
//
// All products are C = A . W^T with A [rows][K] (activations, row-major) and
// W [N][K] (weights stored [out][in]), so both operands are K-contiguous.
//
// bf16 path (bf16 weights, activations as bf16 hi/lo plane pairs): 128x128,
// 64x128 or 64x64 workgroup tiles with K-steps of 64, 4 wave64s in a 2x2
// arrangement, MFMA 16x16x32 bf16 with fp32 accumulate.  Operands are staged
// through LDS (double-buffered, padded row stride) with 16-byte global loads;
// one barrier per K-step; optional deterministic split-K.
// f32 path (small fp32 models): 64x64x16 SIMT tiles.
//
// The row count M is read from device memory so that a launch sized for the
// largest window can be replayed every step; tiles at or past M exit.
#include "bd_internal.h"

#include <math.h>

namespace bd {

static inline int cdiv(int a, int b) { return (a + b - 1) / b; }

__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);   // round to nearest, ties to even
  return (bf16_t)(u >> 16);
}
__device__ __forceinline__ float silu(float x) { return x / (1.0f + expf(-x)); }
// Store x as the bf16 pair (hi at p, lo at p + plane): hi = bf16(x), lo = bf16(x - hi).
__device__ __forceinline__ void store_pair(bf16_t* p, size_t plane, float x) {
  const bf16_t h = f2bf(x);
  p[0] = h;
  p[plane] = f2bf(x - bf2f(h));
}

// ------------------------------------------------------------------ bf16 MFMA
// Activation operands are carried as two bf16 planes, hi = bf16(x) and
// lo = bf16(x - hi), written by the producing kernel; the product is
// accumulated as hi.W + lo.W, two MFMAs per weight fragment, which gives the
// operand 16 significant bits, so that the only activation roundings of the
// forward are the Q/K/V values stored in the KV cache.
constexpr int TBK = 64, LDSK = TBK + 8;

template <int BM, int BN>
struct MfmaTile {
  floatx4 acc[BM / 32][BN / 32];
};

template <int BM, int BN>
struct GemmSmem {
  bf16_t ah[2][BM * LDSK];
  bf16_t al[2][BM * LDSK];
  bf16_t b[2][BN * LDSK];
};

// Main loop over K range [k0, k0 + klen): 4 waves in a 2x2 arrangement, each
// accumulating a (BM/2)x(BN/2) sub-tile of (BM/32)x(BN/32) MFMA tiles.  The
// activation operand comes as two bf16 planes (hi at A, lo at A + a_plane).
template <int BM, int BN>
__device__ __forceinline__ void mfma_mainloop(const bf16_t* __restrict__ A, int lda, size_t a_plane,
                                              const bf16_t* __restrict__ W, int ldw, int k0,
                                              int klen, int m0, int n0, MfmaTile<BM, BN>& t,
                                              GemmSmem<BM, BN>& sm,
                                              const int32_t* __restrict__ arows = nullptr,
                                              int nvalid = 0) {
  constexpr int FM = BM / 32, FN = BN / 32;
  constexpr int CPR = TBK / 8;          // 16-byte chunks per tile row
  constexpr int NA = BM * CPR / 256;    // u32x4 per thread and plane for the A tile
  constexpr int NB = BN * CPR / 256;    // u32x4 per thread for the W tile
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  u32x4 rah[NA], ral[NA];
  u32x4 rb[NB];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) t.acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  // source rows of this thread's A chunks: m0 + r, or a gathered row list
  // (rows past nvalid repeat the first row; their results are discarded)
  const bf16_t* aptr[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int c = tid + 256 * i, r = c / CPR, kc = (c % CPR) * 8;
    const int grow = arows ? arows[r < nvalid ? r : 0] : m0 + r;
    aptr[i] = A + (size_t)grow * lda + kc;
  }

  {
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const bf16_t* src = aptr[i] + k0;
      rah[i] = *(const u32x4*)(src);
      ral[i] = *(const u32x4*)(src + a_plane);
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int c = tid + 256 * i, r = c / CPR, kc = (c % CPR) * 8;
      rb[i] = *(const u32x4*)(W + (size_t)(n0 + r) * ldw + k0 + kc);
    }
  }
  {
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int c = tid + 256 * i, r = c / CPR, kc = (c % CPR) * 8;
      *(u32x4*)(&sm.ah[0][r * LDSK + kc]) = rah[i];
      *(u32x4*)(&sm.al[0][r * LDSK + kc]) = ral[i];
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int c = tid + 256 * i, r = c / CPR, kc = (c % CPR) * 8;
      *(u32x4*)(&sm.b[0][r * LDSK + kc]) = rb[i];
    }
  }
  __syncthreads();
  const int nk = klen / TBK;
  const int arow = wm * (BM / 2) + (lane & 15), brow = wn * (BN / 2) + (lane & 15);
  const int koff = (lane >> 4) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) {
#pragma unroll
      for (int i = 0; i < NA; ++i) {
        const bf16_t* src = aptr[i] + (k0 + (kt + 1) * TBK);
        rah[i] = *(const u32x4*)(src);
        ral[i] = *(const u32x4*)(src + a_plane);
      }
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        const int c = tid + 256 * i, r = c / CPR, kc = (c % CPR) * 8;
        rb[i] = *(const u32x4*)(W + (size_t)(n0 + r) * ldw + (k0 + (kt + 1) * TBK) + kc);
      }
    }
#pragma unroll
    for (int kk = 0; kk < TBK; kk += 32) {
      u32x4 bfr[FN];
#pragma unroll
      for (int j = 0; j < FN; ++j) bfr[j] = *(const u32x4*)(&sm.b[buf][(brow + j * 16) * LDSK + kk + koff]);
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const bf16x8 ah = __builtin_bit_cast(bf16x8, *(const u32x4*)(&sm.ah[buf][(arow + i * 16) * LDSK + kk + koff]));
        const bf16x8 al = __builtin_bit_cast(bf16x8, *(const u32x4*)(&sm.al[buf][(arow + i * 16) * LDSK + kk + koff]));
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const bf16x8 bj = __builtin_bit_cast(bf16x8, bfr[j]);
          t.acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bj, t.acc[i][j], 0, 0, 0);
          t.acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bj, t.acc[i][j], 0, 0, 0);
        }
      }
    }
    if (kt + 1 < nk) {
#pragma unroll
      for (int i = 0; i < NA; ++i) {
        const int c = tid + 256 * i, r = c / CPR, kc = (c % CPR) * 8;
        *(u32x4*)(&sm.ah[buf ^ 1][r * LDSK + kc]) = rah[i];
        *(u32x4*)(&sm.al[buf ^ 1][r * LDSK + kc]) = ral[i];
      }
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        const int c = tid + 256 * i, r = c / CPR, kc = (c % CPR) * 8;
        *(u32x4*)(&sm.b[buf ^ 1][r * LDSK + kc]) = rb[i];
      }
    }
    __syncthreads();
  }
}

// Epilogue modes; with split-K (gridDim.z > 1) every split writes its raw
// partial tile to ws[split][row][col] and k_splitk_reduce applies the mode.
template <int BM, int BN, int EPI>
__global__ __launch_bounds__(256) void k_gemm_bf16(const bf16_t* __restrict__ A, int lda,
                                                   size_t a_plane, const bf16_t* __restrict__ W,
                                                   int ldw, int N, int K,
                                                   const int32_t* __restrict__ Mp,
                                                   void* __restrict__ out, int ldo, size_t out_plane,
                                                   float* __restrict__ ws, int rows_cap) {
  constexpr int FM = BM / 32, FN = BN / 32;
  const int M = *Mp;
  const int m0 = blockIdx.y * BM;
  if (m0 >= M) return;
  const int n0 = blockIdx.x * BN;
  const int splits = gridDim.z, klen = K / splits, k0 = blockIdx.z * klen;
  __shared__ __attribute__((aligned(16))) GemmSmem<BM, BN> sm;
  MfmaTile<BM, BN> t;
  mfma_mainloop<BM, BN>(A, lda, a_plane, W, ldw, k0, klen, m0, n0, t, sm);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + wm * (BM / 2) + i * 16 + (lane >> 4) * 4 + r;
      if (m >= M) continue;
      if (splits > 1) {
        float* wrow = ws + ((size_t)blockIdx.z * rows_cap + m) * N;
#pragma unroll
        for (int j = 0; j < FN; ++j) wrow[n0 + wn * (BN / 2) + j * 16 + (lane & 15)] = t.acc[i][j][r];
      } else if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int j = 0; j < FN; j += 2) {
          const int pb = n0 + wn * (BN / 2) + j * 16;    // packed column of the gate group
          const int col = (pb >> 5) * 16 + (lane & 15);  // output feature
          const float g = t.acc[i][j][r], u = t.acc[i][j + 1][r];
          store_pair((bf16_t*)out + (size_t)m * ldo + col, out_plane, silu(g) * u);
        }
      } else {
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int n = n0 + wn * (BN / 2) + j * 16 + (lane & 15);
          const float v = t.acc[i][j][r];
          if constexpr (EPI == EPI_ADD_F32) ((float*)out)[(size_t)m * ldo + n] += v;
          else ((float*)out)[(size_t)m * ldo + n] = v;
        }
      }
    }
  }
}

// Grouped GEMM over experts: tile ti covers rows [m0, m0 + 128) of expert
// tile_e[ti]; the expert's rows sit at [e_off[e], e_off[e] + e_cnt[e]) of the
// expert-sorted outputs.  The A rows are gathered through a_rows (token rows
// of the expert-sorted assignments) or, with a_rows == NULL, read from the
// expert-sorted layout itself.  W of expert e starts at W + e * w_stride.
template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_grouped(const bf16_t* __restrict__ A, int lda,
                                                      size_t a_plane, const bf16_t* __restrict__ W,
                                                      int ldw, int K, GroupTiles g,
                                                      void* __restrict__ out, int ldo,
                                                      size_t out_plane) {
  constexpr int BM = 128, BN = 128, FM = BM / 32, FN = BN / 32;
  const int ti = blockIdx.y;
  if (ti >= *g.ntiles) return;
  const int e = g.tile_e[ti], m0 = g.tile_m0[ti];
  const int cnt = g.e_cnt[e], base = g.e_off[e];
  const int n0 = blockIdx.x * BN;
  __shared__ __attribute__((aligned(16))) GemmSmem<BM, BN> sm;
  MfmaTile<BM, BN> t;
  const bf16_t* We = W + (size_t)e * g.w_stride;
  if (g.a_rows)
    mfma_mainloop<BM, BN>(A, lda, a_plane, We, ldw, 0, K, 0, n0, t, sm, g.a_rows + base + m0, cnt - m0);
  else
    mfma_mainloop<BM, BN>(A, lda, a_plane, We, ldw, 0, K, base + m0, n0, t, sm);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int ml = m0 + wm * (BM / 2) + i * 16 + (lane >> 4) * 4 + r;
      if (ml >= cnt) continue;
      const size_t orow = (size_t)(base + ml);
      if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int j = 0; j < FN; j += 2) {
          const int pb = n0 + wn * (BN / 2) + j * 16;
          const int col = (pb >> 5) * 16 + (lane & 15);
          store_pair((bf16_t*)out + orow * ldo + col, out_plane, silu(t.acc[i][j][r]) * t.acc[i][j + 1][r]);
        }
      } else {
#pragma unroll
        for (int j = 0; j < FN; ++j)
          ((float*)out)[orow * ldo + n0 + wn * (BN / 2) + j * 16 + (lane & 15)] = t.acc[i][j][r];
      }
    }
  }
}

hipError_t launch_gemm_grouped(int epi, const void* A, int lda, size_t a_plane, const void* W,
                               int ldw, int N, int K, const GroupTiles& g, int max_tiles, void* out,
                               int ldo, size_t out_plane, hipStream_t st) {
  if (N % 128 || K % TBK) return hipErrorInvalidValue;
  dim3 grid(N / 128, max_tiles);
  if (epi == EPI_SWIGLU)
    k_gemm_grouped<EPI_SWIGLU><<<grid, 256, 0, st>>>((const bf16_t*)A, lda, a_plane, (const bf16_t*)W,
                                                     ldw, K, g, out, ldo, out_plane);
  else
    k_gemm_grouped<EPI_STORE_F32><<<grid, 256, 0, st>>>((const bf16_t*)A, lda, a_plane,
                                                        (const bf16_t*)W, ldw, K, g, out, ldo, 0);
  return hipGetLastError();
}

// Deterministic split-K reduction: sums the splits in order, then applies
// the epilogue.  One thread per output element (SwiGLU: per output feature).
template <int EPI>
__global__ __launch_bounds__(256) void k_splitk_reduce(const float* __restrict__ ws, int splits,
                                                       int N, int rows_cap,
                                                       const int32_t* __restrict__ Mp,
                                                       void* __restrict__ out, int ldo,
                                                       size_t out_plane) {
  const int M = *Mp;
  const int ncols = (EPI == EPI_SWIGLU) ? N / 2 : N;
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int m = (int)(idx / ncols), c = (int)(idx % ncols);
  if (m >= M) return;
  if constexpr (EPI == EPI_SWIGLU) {
    const int pg = (c >> 4) * 32 + (c & 15);
    float g = 0.f, u = 0.f;
    for (int z = 0; z < splits; ++z) {
      const float* w = ws + ((size_t)z * rows_cap + m) * N;
      g += w[pg];
      u += w[pg + 16];
    }
    store_pair((bf16_t*)out + (size_t)m * ldo + c, out_plane, silu(g) * u);
  } else {
    float v = 0.f;
    for (int z = 0; z < splits; ++z) v += ws[((size_t)z * rows_cap + m) * N + c];
    if constexpr (EPI == EPI_ADD_F32) ((float*)out)[(size_t)m * ldo + c] += v;
    else ((float*)out)[(size_t)m * ldo + c] = v;
  }
}

// Fused LM head: for its 128 vocabulary columns the workgroup reduces each row
// to (max z, sum exp(z - max), lowest argmax) and writes one partial per
// (column tile, row); logits never leave registers.
__global__ __launch_bounds__(256) void k_lm_head_bf16(const bf16_t* __restrict__ A, int d,
                                                      size_t a_plane,
                                                      const bf16_t* __restrict__ W, int mask_id,
                                                      float scale, const int32_t* __restrict__ Mp,
                                                      int rows_cap, float* __restrict__ pmax,
                                                      float* __restrict__ psum,
                                                      int32_t* __restrict__ parg) {
  constexpr int TBM = 128, TBN = 128;
  const int M = *Mp;
  const int m0 = blockIdx.y * TBM;
  if (m0 >= M) return;
  const int n0 = blockIdx.x * TBN;
  __shared__ __attribute__((aligned(16))) GemmSmem<TBM, TBN> sm;
  __shared__ float red_m[2][TBM], red_s[2][TBM];
  __shared__ int32_t red_a[2][TBM];
  MfmaTile<TBM, TBN> t;
  mfma_mainloop<TBM, TBN>(A, d, a_plane, W, d, 0, d, m0, n0, t, sm);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float v[4];
      float mx = -INFINITY;
      int arg = 0x7fffffff;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int n = n0 + wn * 64 + j * 16 + (lane & 15);
        v[j] = (n == mask_id) ? -INFINITY : scale * t.acc[i][j][r];
        if (v[j] > mx) { mx = v[j]; arg = n; }
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) {
        const float om = __shfl_xor(mx, off);
        const int oa = __shfl_xor(arg, off);
        if (om > mx || (om == mx && oa < arg)) { mx = om; arg = oa; }
      }
      float s = 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) s += expf(v[j] - mx);
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) s += __shfl_xor(s, off);
      if ((lane & 15) == 0) {
        const int rl = wm * 64 + i * 16 + (lane >> 4) * 4 + r;
        red_m[wn][rl] = mx;
        red_s[wn][rl] = s;
        red_a[wn][rl] = arg;
      }
    }
  }
  __syncthreads();
  if (threadIdx.x < TBM) {
    const int rl = threadIdx.x, m = m0 + rl;
    if (m < M) {
      const float ma = red_m[0][rl], mb = red_m[1][rl];
      const float mm = fmaxf(ma, mb);
      const float s = red_s[0][rl] * expf(ma - mm) + red_s[1][rl] * expf(mb - mm);
      const int a = (ma >= mb) ? red_a[0][rl] : red_a[1][rl];
      const size_t o = (size_t)blockIdx.x * rows_cap + m;
      pmax[o] = mm;
      psum[o] = s;
      parg[o] = a;
    }
  }
}

// ------------------------------------------------------------------ f32 SIMT
constexpr int SBM = 64, SBN = 64, SBK = 16;

__device__ __forceinline__ void simt_mainloop(const float* __restrict__ A, int lda,
                                              const float* __restrict__ W, int ldw, int K, int m0,
                                              int n0, float acc[4][4], float* sA, float* sB) {
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
  for (int k0 = 0; k0 < K; k0 += SBK) {
    // 64 rows x 16 k = 1024 floats per operand: 4 per thread
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int c = tid + 256 * q, r = c >> 4, kk = c & 15;
      sA[kk * (SBM + 1) + r] = A[(size_t)(m0 + r) * lda + k0 + kk];
      sB[kk * (SBN + 1) + r] = W[(size_t)(n0 + r) * ldw + k0 + kk];
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < SBK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = sA[kk * (SBM + 1) + ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = sB[kk * (SBN + 1) + tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
}

template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_f32(const float* __restrict__ A, int lda,
                                                  const float* __restrict__ W, int ldw, int N, int K,
                                                  const int32_t* __restrict__ Mp,
                                                  void* __restrict__ out, int ldo) {
  const int M = *Mp;
  const int m0 = blockIdx.y * SBM;
  if (m0 >= M) return;
  const int n0 = blockIdx.x * SBN;
  __shared__ float sA[SBK * (SBM + 1)], sB[SBK * (SBN + 1)];
  float acc[4][4];
  simt_mainloop(A, lda, W, ldw, K, m0, n0, acc, sA, sB);
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= M) continue;
    if constexpr (EPI == EPI_SWIGLU) {
      // packed gate/up groups of 16 columns: j even = gate, j odd = up
#pragma unroll
      for (int j = 0; j < 4; j += 2) {
        const int pb = n0 + 16 * j;
        const int col = (pb >> 5) * 16 + tx;
        ((float*)out)[(size_t)m * ldo + col] = silu(acc[i][j]) * acc[i][j + 1];
      }
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int n = n0 + tx + 16 * j;
        if constexpr (EPI == EPI_ADD_F32) ((float*)out)[(size_t)m * ldo + n] += acc[i][j];
        else ((float*)out)[(size_t)m * ldo + n] = acc[i][j];
      }
    }
  }
}

__global__ __launch_bounds__(256) void k_lm_head_f32(const float* __restrict__ A, int d,
                                                     const float* __restrict__ W, int mask_id,
                                                     float scale, const int32_t* __restrict__ Mp,
                                                     int rows_cap, float* __restrict__ pmax,
                                                     float* __restrict__ psum,
                                                     int32_t* __restrict__ parg) {
  const int M = *Mp;
  const int m0 = blockIdx.y * SBM;
  if (m0 >= M) return;
  const int n0 = blockIdx.x * SBN;
  __shared__ float sA[SBK * (SBM + 1)], sB[SBK * (SBN + 1)];
  float acc[4][4];
  simt_mainloop(A, d, W, d, d, m0, n0, acc, sA, sB);
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float v[4], mx = -INFINITY;
    int arg = 0x7fffffff;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx + 16 * j;
      v[j] = (n == mask_id) ? -INFINITY : scale * acc[i][j];
      if (v[j] > mx || (v[j] == mx && n < arg)) { mx = v[j]; arg = n; }
    }
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
      const float om = __shfl_xor(mx, off);
      const int oa = __shfl_xor(arg, off);
      if (om > mx || (om == mx && oa < arg)) { mx = om; arg = oa; }
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) s += expf(v[j] - mx);
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) s += __shfl_xor(s, off);
    const int m = m0 + ty * 4 + i;
    if (tx == 0 && m < M) {
      const size_t o = (size_t)blockIdx.x * rows_cap + m;
      pmax[o] = mx;
      psum[o] = s;
      parg[o] = arg;
    }
  }
}

// Merge the per-tile partials of each row (one wave per row, deterministic):
// max and lowest argmax over tiles, then sum_t s_t exp(m_t - max) with a
// fixed lane assignment and a fixed shuffle tree; conf = 1 / sum.
__global__ __launch_bounds__(256) void k_lm_merge(const float* __restrict__ pmax,
                                                  const float* __restrict__ psum,
                                                  const int32_t* __restrict__ parg, int ntiles,
                                                  const int32_t* __restrict__ Mp, int rows_cap,
                                                  float* __restrict__ conf, int32_t* __restrict__ tok) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int m = blockIdx.x * 4 + wave;
  if (m >= *Mp) return;
  float mx = -INFINITY;
  int arg = 0x7fffffff;
  for (int t = lane; t < ntiles; t += 64) {
    const float v = pmax[(size_t)t * rows_cap + m];
    const int a = parg[(size_t)t * rows_cap + m];
    if (v > mx || (v == mx && a < arg)) { mx = v; arg = a; }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const float om = __shfl_xor(mx, off);
    const int oa = __shfl_xor(arg, off);
    if (om > mx || (om == mx && oa < arg)) { mx = om; arg = oa; }
  }
  float s = 0.f;
  for (int t = lane; t < ntiles; t += 64) {
    const size_t o = (size_t)t * rows_cap + m;
    s += psum[o] * expf(pmax[o] - mx);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  if (lane == 0) {
    conf[m] = 1.0f / s;
    tok[m] = arg;
  }
}

// ------------------------------------------------------------------ launchers

template <int BM, int BN>
static void launch_bf16_cfg(int epi, dim3 grid, const bf16_t* a, int lda, size_t ap, const bf16_t* w,
                            int ldw, int N, int K, const int32_t* M_dev, void* o, int ldo, size_t op,
                            float* ws, int rows_cap, hipStream_t st) {
  switch (epi) {
    case EPI_ADD_F32:
      k_gemm_bf16<BM, BN, EPI_ADD_F32><<<grid, 256, 0, st>>>(a, lda, ap, w, ldw, N, K, M_dev, o, ldo, op, ws, rows_cap);
      break;
    case EPI_SWIGLU:
      k_gemm_bf16<BM, BN, EPI_SWIGLU><<<grid, 256, 0, st>>>(a, lda, ap, w, ldw, N, K, M_dev, o, ldo, op, ws, rows_cap);
      break;
    default:
      k_gemm_bf16<BM, BN, EPI_STORE_F32><<<grid, 256, 0, st>>>(a, lda, ap, w, ldw, N, K, M_dev, o, ldo, op, ws, rows_cap);
      break;
  }
}

// Tile choice: the largest tile that still gives >= 512 workgroups over the
// row capacity; otherwise 64x64 tiles with a deterministic split-K (each
// split at least 512 deep, workspace permitting) to reach that count.
GemmPlan plan_gemm(bool is_bf16, int N, int K, int rows_cap) {
  GemmPlan p{64, 64, 1};
  if (!is_bf16) return p;
  const int target = 512;
  const int cand[3][2] = {{128, 128}, {64, 128}, {64, 64}};
  for (auto& c : cand) {
    if (N % c[1]) continue;
    const int wgs = (N / c[1]) * cdiv(rows_cap, c[0]);
    if (wgs >= target) return GemmPlan{c[0], c[1], 1};
  }
  const int wgs = (N / 64) * cdiv(rows_cap, 64);
  int splits = 1;
  while (wgs * splits < target && K % (2 * splits * TBK) == 0 && K / (2 * splits) >= 512) splits *= 2;
  return GemmPlan{64, 64, splits};
}

size_t gemm_workspace_floats(const GemmPlan& p, int N, int rows_cap) {
  return p.splits > 1 ? (size_t)p.splits * rows_cap * N : 0;
}

hipError_t launch_gemm(int epi, bool is_bf16, const void* A, int lda, size_t a_plane, const void* W,
                       int ldw, int N, int K, const int32_t* M_dev, int rows_cap, void* out, int ldo,
                       size_t out_plane, float* ws, size_t ws_floats, hipStream_t st) {
  if (is_bf16) {
    GemmPlan p = plan_gemm(true, N, K, rows_cap);
    if (gemm_workspace_floats(p, N, rows_cap) > ws_floats || !ws) p.splits = 1;
    if (N % p.bn || K % (TBK * p.splits)) return hipErrorInvalidValue;
    dim3 grid(N / p.bn, cdiv(rows_cap, p.bm), p.splits);
    const bf16_t* a = (const bf16_t*)A;
    const bf16_t* w = (const bf16_t*)W;
    if (p.bm == 128) launch_bf16_cfg<128, 128>(epi, grid, a, lda, a_plane, w, ldw, N, K, M_dev, out, ldo, out_plane, ws, rows_cap, st);
    else if (p.bn == 128) launch_bf16_cfg<64, 128>(epi, grid, a, lda, a_plane, w, ldw, N, K, M_dev, out, ldo, out_plane, ws, rows_cap, st);
    else launch_bf16_cfg<64, 64>(epi, grid, a, lda, a_plane, w, ldw, N, K, M_dev, out, ldo, out_plane, ws, rows_cap, st);
    if (p.splits > 1) {
      const int ncols = epi == EPI_SWIGLU ? N / 2 : N;
      const size_t total = (size_t)rows_cap * ncols;
      const int blocks = (int)((total + 255) / 256);
      switch (epi) {
        case EPI_ADD_F32: k_splitk_reduce<EPI_ADD_F32><<<blocks, 256, 0, st>>>(ws, p.splits, N, rows_cap, M_dev, out, ldo, out_plane); break;
        case EPI_SWIGLU: k_splitk_reduce<EPI_SWIGLU><<<blocks, 256, 0, st>>>(ws, p.splits, N, rows_cap, M_dev, out, ldo, out_plane); break;
        default: k_splitk_reduce<EPI_STORE_F32><<<blocks, 256, 0, st>>>(ws, p.splits, N, rows_cap, M_dev, out, ldo, out_plane); break;
      }
    }
  } else {
    if (N % SBN || K % SBK) return hipErrorInvalidValue;
    dim3 grid(N / SBN, cdiv(rows_cap, SBM));
    const float* a = (const float*)A;
    const float* w = (const float*)W;
    switch (epi) {
      case EPI_ADD_F32: k_gemm_f32<EPI_ADD_F32><<<grid, 256, 0, st>>>(a, lda, w, ldw, N, K, M_dev, out, ldo); break;
      case EPI_SWIGLU: k_gemm_f32<EPI_SWIGLU><<<grid, 256, 0, st>>>(a, lda, w, ldw, N, K, M_dev, out, ldo); break;
      default: k_gemm_f32<EPI_STORE_F32><<<grid, 256, 0, st>>>(a, lda, w, ldw, N, K, M_dev, out, ldo); break;
    }
  }
  return hipGetLastError();
}

hipError_t launch_lm_head(bool is_bf16, const void* A, int d, size_t a_plane, const void* W, int V,
                          int mask_id, float scale, const int32_t* M_dev, int rows_cap,
                          float* part_max,
                          float* part_sum, int32_t* part_arg, float* conf, int32_t* tok,
                          hipStream_t st) {
  int ntiles;
  if (is_bf16) {
    if (V % 128 || d % TBK) return hipErrorInvalidValue;
    ntiles = V / 128;
    dim3 grid(ntiles, cdiv(rows_cap, 128));
    k_lm_head_bf16<<<grid, 256, 0, st>>>((const bf16_t*)A, d, a_plane, (const bf16_t*)W, mask_id, scale, M_dev,
                                        rows_cap, part_max, part_sum, part_arg);
  } else {
    if (V % SBN || d % SBK) return hipErrorInvalidValue;
    ntiles = V / SBN;
    dim3 grid(ntiles, cdiv(rows_cap, SBM));
    k_lm_head_f32<<<grid, 256, 0, st>>>((const float*)A, d, (const float*)W, mask_id, scale, M_dev,
                                       rows_cap, part_max, part_sum, part_arg);
  }
  k_lm_merge<<<cdiv(rows_cap, 4), 256, 0, st>>>(part_max, part_sum, part_arg, ntiles, M_dev, rows_cap,
                                                conf, tok);
  return hipGetLastError();
}

__global__ void k_logits_post(float* __restrict__ z, int V, int mask_id, float scale,
                              const int32_t* __restrict__ Mp) {
  const int m = blockIdx.y;
  if (m >= *Mp) return;
  for (int n = blockIdx.x * blockDim.x + threadIdx.x; n < V; n += gridDim.x * blockDim.x) {
    float& v = z[(size_t)m * V + n];
    v = (n == mask_id) ? -INFINITY : scale * v;
  }
}

hipError_t launch_lm_logits(bool is_bf16, const void* A, int d, size_t a_plane, const void* W, int V,
                            int mask_id, float scale, const int32_t* M_dev, int rows_cap,
                            float* logits, hipStream_t st) {
  hipError_t e = launch_gemm(EPI_STORE_F32, is_bf16, A, d, a_plane, W, d, V, d, M_dev, rows_cap,
                             logits, V, 0, nullptr, 0, st);
  if (e != hipSuccess) return e;
  k_logits_post<<<dim3(cdiv(V, 256 * 8), rows_cap), 256, 0, st>>>(logits, V, mask_id, scale, M_dev);
  return hipGetLastError();
}

}  // namespace bd
