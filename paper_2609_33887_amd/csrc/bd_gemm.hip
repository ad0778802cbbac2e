// Projection GEMMs and the fused LM-head softmax-statistics kernel.
//
// All products are C = A . W^T with A [rows][K] (activations, row-major) and
// W [N][K] (weights stored [out][in]), so both operands are K-contiguous.
//
// bf16 path (bf16 weights, fp32 activations): 128x128x32 workgroup tiles,
// 4 wave64s in a 2x2 arrangement each owning a 64x64 sub-tile of 4x4 MFMA
// 16x16x32 bf16 tiles (fp32 accumulate).  Operands are staged through LDS
// (double-buffered, padded row stride) with 16-byte global loads; one barrier
// per K-step.
// f32 path (small fp32 models): 64x64x16 SIMT tiles.
//
// The row count M is read from device memory so that a launch sized for the
// largest window can be replayed every step; tiles at or past M exit.
#include "bd_internal.h"

#include <math.h>

namespace bd {

__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);   // round to nearest, ties to even
  return (bf16_t)(u >> 16);
}
__device__ __forceinline__ float silu(float x) { return x / (1.0f + expf(-x)); }

// ------------------------------------------------------------------ bf16 MFMA
// Activations are fp32 in memory.  While staging a tile into LDS each value
// x is split into hi = bf16(x) and lo = bf16(x - hi), and the product is
// accumulated as hi.W + lo.W: two MFMAs per weight fragment give the
// activation operand 16 significant bits, so that the only activation
// roundings of the forward are the Q/K/V values stored in the KV cache.
constexpr int TBM = 128, TBN = 128, TBK = 32, LDSK = TBK + 8;

struct MfmaTile {
  floatx4 acc[4][4];
};

struct GemmSmem {
  bf16_t ah[2][TBM * LDSK];
  bf16_t al[2][TBM * LDSK];
  bf16_t b[2][TBN * LDSK];
};

__device__ __forceinline__ void split4(float4 v, uint2& hi, uint2& lo) {
  const float x[4] = {v.x, v.y, v.z, v.w};
  bf16_t h[4], l[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    h[e] = f2bf(x[e]);
    l[e] = f2bf(x[e] - bf2f(h[e]));
  }
  hi = make_uint2((uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16));
  lo = make_uint2((uint32_t)l[0] | ((uint32_t)l[1] << 16), (uint32_t)l[2] | ((uint32_t)l[3] << 16));
}

// Main loop: accumulates the 64x64 sub-tile of this wave.
__device__ __forceinline__ void mfma_mainloop(const float* __restrict__ A, int lda,
                                              const bf16_t* __restrict__ W, int ldw, int K, int m0,
                                              int n0, MfmaTile& t, GemmSmem& sm) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  float4 ra[4];
  uint4 rb[2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) t.acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  // A tile: 128 rows x 32 fp32 = 1024 float4 (4 per thread);
  // W tile: 128 rows x 32 bf16 = 512 uint4 (2 per thread).
#define GLOAD(k0)                                                                    \
  do {                                                                               \
    _Pragma("unroll") for (int i = 0; i < 4; ++i) {                                  \
      const int c = tid + 256 * i, r = c >> 3, kc = (c & 7) * 4;                     \
      ra[i] = *(const float4*)(A + (size_t)(m0 + r) * lda + (k0) + kc);              \
    }                                                                                \
    _Pragma("unroll") for (int i = 0; i < 2; ++i) {                                  \
      const int c = tid + 256 * i, r = c >> 2, kc = (c & 3) * 8;                     \
      rb[i] = *(const uint4*)(W + (size_t)(n0 + r) * ldw + (k0) + kc);               \
    }                                                                                \
  } while (0)
#define SSTORE(buf)                                                                  \
  do {                                                                               \
    _Pragma("unroll") for (int i = 0; i < 4; ++i) {                                  \
      const int c = tid + 256 * i, r = c >> 3, kc = (c & 7) * 4;                     \
      uint2 hi, lo;                                                                  \
      split4(ra[i], hi, lo);                                                         \
      *(uint2*)(&sm.ah[buf][r * LDSK + kc]) = hi;                                    \
      *(uint2*)(&sm.al[buf][r * LDSK + kc]) = lo;                                    \
    }                                                                                \
    _Pragma("unroll") for (int i = 0; i < 2; ++i) {                                  \
      const int c = tid + 256 * i, r = c >> 2, kc = (c & 3) * 8;                     \
      *(uint4*)(&sm.b[buf][r * LDSK + kc]) = rb[i];                                  \
    }                                                                                \
  } while (0)

  GLOAD(0);
  SSTORE(0);
  __syncthreads();
  const int nk = K / TBK;
  const int arow = wm * 64 + (lane & 15), brow = wn * 64 + (lane & 15), koff = (lane >> 4) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) GLOAD((kt + 1) * TBK);
    bf16x8 ah[4], al[4], bfr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ah[i] = *(const bf16x8*)(&sm.ah[buf][(arow + i * 16) * LDSK + koff]);
      al[i] = *(const bf16x8*)(&sm.al[buf][(arow + i * 16) * LDSK + koff]);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) bfr[j] = *(const bf16x8*)(&sm.b[buf][(brow + j * 16) * LDSK + koff]);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        t.acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[i], bfr[j], t.acc[i][j], 0, 0, 0);
        t.acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[i], bfr[j], t.acc[i][j], 0, 0, 0);
      }
    if (kt + 1 < nk) SSTORE(buf ^ 1);
    __syncthreads();
  }
#undef GLOAD
#undef SSTORE
}

template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_bf16(const float* __restrict__ A, int lda,
                                                   const bf16_t* __restrict__ W, int ldw, int N, int K,
                                                   const int32_t* __restrict__ Mp,
                                                   float* __restrict__ out, int ldo) {
  const int M = *Mp;
  const int m0 = blockIdx.y * TBM;
  if (m0 >= M) return;
  const int n0 = blockIdx.x * TBN;
  __shared__ __attribute__((aligned(16))) GemmSmem sm;
  MfmaTile t;
  mfma_mainloop(A, lda, W, ldw, K, m0, n0, t, sm);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + wm * 64 + i * 16 + (lane >> 4) * 4 + r;
      if (m >= M) continue;
      if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int j = 0; j < 4; j += 2) {
          const int pb = n0 + wn * 64 + j * 16;          // packed column of the gate group
          const int col = (pb >> 5) * 16 + (lane & 15);  // output feature
          const float g = t.acc[i][j][r], u = t.acc[i][j + 1][r];
          out[(size_t)m * ldo + col] = silu(g) * u;
        }
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = n0 + wn * 64 + j * 16 + (lane & 15);
          const float v = t.acc[i][j][r];
          if constexpr (EPI == EPI_ADD_F32) out[(size_t)m * ldo + n] += v;
          else out[(size_t)m * ldo + n] = v;
        }
      }
    }
  }
}

// Fused LM head: for its 128 vocabulary columns the workgroup reduces each row
// to (max z, sum exp(z - max), lowest argmax) and writes one partial per
// (column tile, row); logits never leave registers.
__global__ __launch_bounds__(256) void k_lm_head_bf16(const float* __restrict__ A, int d,
                                                      const bf16_t* __restrict__ W, int mask_id,
                                                      float scale, const int32_t* __restrict__ Mp,
                                                      int rows_cap, float* __restrict__ pmax,
                                                      float* __restrict__ psum,
                                                      int32_t* __restrict__ parg) {
  const int M = *Mp;
  const int m0 = blockIdx.y * TBM;
  if (m0 >= M) return;
  const int n0 = blockIdx.x * TBN;
  __shared__ __attribute__((aligned(16))) GemmSmem sm;
  __shared__ float red_m[2][TBM], red_s[2][TBM];
  __shared__ int32_t red_a[2][TBM];
  MfmaTile t;
  mfma_mainloop(A, d, W, d, d, m0, n0, t, sm);
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

// Merge the per-tile partials of each row in tile order (deterministic):
// conf = 1 / sum_t s_t exp(m_t - max), tok = lowest index attaining the max.
__global__ __launch_bounds__(256) void k_lm_merge(const float* __restrict__ pmax,
                                                  const float* __restrict__ psum,
                                                  const int32_t* __restrict__ parg, int ntiles,
                                                  const int32_t* __restrict__ Mp, int rows_cap,
                                                  float* __restrict__ conf, int32_t* __restrict__ tok) {
  const int M = *Mp;
  const int m = blockIdx.x * blockDim.x + threadIdx.x;
  if (m >= M) return;
  float mx = -INFINITY;
  int arg = 0;
  for (int t = 0; t < ntiles; ++t) {
    const float v = pmax[(size_t)t * rows_cap + m];
    if (v > mx) { mx = v; arg = parg[(size_t)t * rows_cap + m]; }
  }
  float s = 0.f;
  for (int t = 0; t < ntiles; ++t) {
    const size_t o = (size_t)t * rows_cap + m;
    s += psum[o] * expf(pmax[o] - mx);
  }
  conf[m] = 1.0f / s;
  tok[m] = arg;
}

// ------------------------------------------------------------------ launchers
static inline int cdiv(int a, int b) { return (a + b - 1) / b; }

hipError_t launch_gemm(int epi, bool is_bf16, const void* A, int lda, const void* W, int ldw, int N,
                       int K, const int32_t* M_dev, int rows_cap, void* out, int ldo,
                       hipStream_t st) {
  if (is_bf16) {
    if (N % TBN || K % TBK) return hipErrorInvalidValue;
    dim3 grid(N / TBN, cdiv(rows_cap, TBM));
    const float* a = (const float*)A;
    const bf16_t* w = (const bf16_t*)W;
    float* o = (float*)out;
    switch (epi) {
      case EPI_ADD_F32: k_gemm_bf16<EPI_ADD_F32><<<grid, 256, 0, st>>>(a, lda, w, ldw, N, K, M_dev, o, ldo); break;
      case EPI_SWIGLU: k_gemm_bf16<EPI_SWIGLU><<<grid, 256, 0, st>>>(a, lda, w, ldw, N, K, M_dev, o, ldo); break;
      default: k_gemm_bf16<EPI_STORE_F32><<<grid, 256, 0, st>>>(a, lda, w, ldw, N, K, M_dev, o, ldo); break;
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

hipError_t launch_lm_head(bool is_bf16, const void* A, int d, const void* W, int V, int mask_id,
                          float scale, const int32_t* M_dev, int rows_cap, float* part_max,
                          float* part_sum, int32_t* part_arg, float* conf, int32_t* tok,
                          hipStream_t st) {
  int ntiles;
  if (is_bf16) {
    if (V % TBN || d % TBK) return hipErrorInvalidValue;
    ntiles = V / TBN;
    dim3 grid(ntiles, cdiv(rows_cap, TBM));
    k_lm_head_bf16<<<grid, 256, 0, st>>>((const float*)A, d, (const bf16_t*)W, mask_id, scale, M_dev,
                                        rows_cap, part_max, part_sum, part_arg);
  } else {
    if (V % SBN || d % SBK) return hipErrorInvalidValue;
    ntiles = V / SBN;
    dim3 grid(ntiles, cdiv(rows_cap, SBM));
    k_lm_head_f32<<<grid, 256, 0, st>>>((const float*)A, d, (const float*)W, mask_id, scale, M_dev,
                                       rows_cap, part_max, part_sum, part_arg);
  }
  k_lm_merge<<<cdiv(rows_cap, 256), 256, 0, st>>>(part_max, part_sum, part_arg, ntiles, M_dev, rows_cap,
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

hipError_t launch_lm_logits(bool is_bf16, const void* A, int d, const void* W, int V, int mask_id,
                            float scale, const int32_t* M_dev, int rows_cap, float* logits,
                            hipStream_t st) {
  hipError_t e = launch_gemm(EPI_STORE_F32, is_bf16, A, d, W, d, V, d, M_dev, rows_cap, logits, V, st);
  if (e != hipSuccess) return e;
  k_logits_post<<<dim3(cdiv(V, 256 * 8), rows_cap), 256, 0, st>>>(logits, V, mask_id, scale, M_dev);
  return hipGetLastError();
}

}  // namespace bd
