// Projection GEMMs and the fused LM-head softmax-statistics kernel.
//
// All products are C = A . W^T with A [rows][K] (activations, row-major) and
// W [N][K] (weights stored [out][in]), so both operands are K-contiguous.
//
// bf16 path (bf16 weights, activations as bf16 hi/lo plane pairs): workgroup
// tiles of 128x256 (8 wave64s of 64x64), 128x128 (4 waves of 64x64, or 8 of
// 64x32), 64x128 (4 waves of 32x64) or 64x64 (4 waves of 32x32), the waves
// in a 2 x (waves / 2)
// arrangement, MFMA 16x16x32 bf16 with fp32 accumulate (plan_gemm and the
// launchers choose).  Operands reach LDS through direct global-to-LDS loads
// into a four-stage ring (K-stages of 32, swizzled rows); one barrier per
// stage; the residual projections may split K (the partial sums are folded
// in by the next RMSNorm).
// fp8 weights (WQ = WQ_FP8): W holds OCP fp8 E4M3 codes, one byte per
// element, with a power-of-two scale per output row; the W stage holds
// 32-byte rows, each lane converts its 8 codes of a fragment to bf16 (exact)
// before the MFMA, and the epilogue multiplies each output column by its row
// scale (exact, so the result equals the bf16 product with the dequantized
// weights).
// MXFP4 weights (WQ = WQ_MXFP4): a 32-deep stage is one MX block, so the
// stage holds each W row's 16 bytes of E2M1 codes and its block exponent; the
// lane converts its 8 codes with the block scale (v_cvt_scalef32_pk_bf16_fp4:
// E2M1 value x 2^X, exact in bf16), again the bf16 product with the
// dequantized weights.  The codes are stored stage-major (WQuant), so a
// stage's W rows are one contiguous run of 16-byte rows.
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
//
// Main loop: K advances in stages of SK = 32 through a ring of four LDS
// stages filled by direct buffer-to-LDS 16-byte loads (no register staging,
// no LDS store instructions); three stages are in flight while the fourth is
// consumed, and one barrier per stage both publishes the stage and retires
// the one the next loads overwrite.  The bf16 operands go through buffer
// resources rather than global (flat) addresses: the compiler counts a flat
// load into LDS as pending LDS traffic too, which turned every LDS wait of
// the loop into a full drain; with buffer loads the waits count the
// fragment reads down, and the 32-bit lane offsets replace 64-bit address
// arithmetic (130 instead of 152 VGPRs in the 128x256 tile).  A wave's load
// instruction writes 1 KiB of LDS = 16 rows x 64 B, lane l at byte 16 l; in
// LDS the 16-byte chunk c of row r sits at position c ^ swz(r),
// swz(r) = (r >> 1) & 3.  A fragment read (lane l: row l & 15, chunk l >> 4)
// is then free of bank conflicts: measured with
// the LDS bank-conflict counter on gfx950, this pattern reads 141 B/clk per CU
// with no conflict cycles, where the earlier (r >> 1) & 3 ^ (r >> 3) & 1 had
// two-way conflicts (106 B/clk) and unswizzled rows 114 B/clk.
constexpr int SK = 32;       // K per pipeline stage (KALIGN = 4 stages)

__device__ __forceinline__ int swz(int r) { return (r >> 1) & 3; }

typedef __attribute__((address_space(3))) void lds_void_t;

// Fourth word of a raw buffer resource on gfx9-family parts: 32-bit data
// format (a zero format reads zeros), no index stride, no swizzle.
constexpr int BUF_DWORD3 = 0x00020000;

template <int BM, int BN, int WQ = WQ_NONE>
struct GemmStage {
  bf16_t ah[BM * SK];
  bf16_t al[BM * SK];
  // bf16 rows of 64 B, fp8 rows of 32 B, or E2M1 rows of 16 B
  bf16_t b[WQ == WQ_NONE ? BN * SK : (WQ == WQ_FP8 ? BN * SK / 2 : BN * SK / 4)];
  uint8_t be[WQ == WQ_MXFP4 ? BN : 0];    // the MXFP4 rows' block exponents
};

// fp8 W loads per wave and stage: BN = 128 -> one 16-byte load per lane
// (32 rows of 32 B per wave); BN = 64 -> two 4-byte loads (8 rows each).
template <int BN>
struct W8Load {
  static constexpr int bytes = BN == 128 ? 16 : 4;
  static constexpr int loads = BN * SK / (4 * 64 * bytes);
  static constexpr int rows = 64 * bytes / SK;      // rows per load instruction
};

// MXFP4 W loads per wave and stage: BN rows x 16 B of codes as 4-byte loads
// (16 rows per load instruction), plus one 4-byte load of BN / 4 exponents.
template <int BN>
struct W4Load {
  static constexpr int loads = BN * 16 / (4 * 64 * 4);
};

// Eight E2M1 codes (nibbles of v, k order, low nibble first) times the block
// scale -> eight bf16 (exact).
__device__ __forceinline__ bf16x8 fp4x8_to_bf16(uint32_t v, float scale) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(v, scale, 0);
  const bf16x2_t b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(v, scale, 1);
  const bf16x2_t c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(v, scale, 2);
  const bf16x2_t d = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(v, scale, 3);
  bf16x8 o;
  o[0] = a[0]; o[1] = a[1]; o[2] = b[0]; o[3] = b[1];
  o[4] = c[0]; o[5] = c[1]; o[6] = d[0]; o[7] = d[1];
  return o;
}

// Eight E4M3 codes (bytes 0..7 of v, k order) -> eight bf16 (exact).
__device__ __forceinline__ bf16x8 fp8x8_to_bf16(uint2 v) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(v.x, 1.0f, false);
  const bf16x2_t b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(v.x, 1.0f, true);
  const bf16x2_t c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(v.y, 1.0f, false);
  const bf16x2_t d = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(v.y, 1.0f, true);
  bf16x8 o;
  o[0] = a[0]; o[1] = a[1]; o[2] = b[0]; o[3] = b[1];
  o[4] = c[0]; o[5] = c[1]; o[6] = d[0]; o[7] = d[1];
  return o;
}

// NW waves per workgroup in a 2 x (NW / 2) arrangement: each wave owns
// (BM / 2) x (2 BN / NW) of the tile.
template <int BM, int BN, int NW = 4>
struct MfmaTile {
  floatx4 acc[BM / 32][BN / (8 * NW)];
};

// s_waitcnt vmcnt(N) lgkmcnt(0) (gfx9 encoding): before a stage barrier the
// wave's global->LDS loads but the N youngest have landed and all of its LDS
// reads have returned, so that no wave overwrites a stage another still
// reads (the barrier itself waits for neither)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (0 << 8));
}

// Per-thread sources of one tile's loads: the lane's 16-byte chunk of its A
// rows (hi and lo planes) and W rows, as byte offsets into buffer resources
// for A and bf16 W, as pointers for quantized W.
template <int BM, int BN, int WQ = WQ_NONE, int NW = 4>
struct TileSrc {
  // A planes and bf16 W through buffer resources (the range check off): the
  // lane's byte offset from the resource base; the stage adds 2 k bytes
  __amdgpu_buffer_rsrc_t ra_h, ra_l, rw;
  uint32_t a[BM / (16 * NW)];
  uint32_t w[WQ == WQ_NONE ? BN / (16 * NW) : 1];
  const uint8_t* w8[WQ == WQ_FP8 ? W8Load<BN>::loads : 1];
  const uint8_t* w4[WQ == WQ_MXFP4 ? W4Load<BN>::loads : 1];
  const uint8_t* we;        // MXFP4: this lane's 4 exponents of the first stage
  size_t kstep;             // MXFP4: rows per stage block (codes advance 16 bytes a row)
};

template <int BM, int BN, int WQ, int NW = 4>
__device__ __forceinline__ void stage_issue(const TileSrc<BM, BN, WQ, NW>& src, size_t a_plane, int k,
                                            GemmStage<BM, BN, WQ>& s, int wave) {
  static_assert(WQ == WQ_NONE || NW == 4, "quantized weights take four waves");
#pragma unroll
  for (int i = 0; i < BM / (16 * NW); ++i) {
    const int r = (i * NW + wave) * 16;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(src.ra_h, (lds_void_t*)(s.ah + r * SK), 16, src.a[i], 2 * k, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(src.ra_l, (lds_void_t*)(s.al + r * SK), 16, src.a[i], 2 * k, 0, 0);
  }
  if constexpr (WQ == WQ_FP8) {
    typedef W8Load<BN> L;
    uint8_t* b8 = (uint8_t*)s.b;
#pragma unroll
    for (int i = 0; i < L::loads; ++i) {
      const int r = (wave * L::loads + i) * L::rows;
      __builtin_amdgcn_global_load_lds((const void*)(src.w8[i] + k), (lds_void_t*)(b8 + r * SK), L::bytes, 0, 0);
    }
  } else if constexpr (WQ == WQ_MXFP4) {
    // stage k is block k / SK: codes advance kstep rows of 16 bytes a block,
    // exponents kstep bytes; wave w fills 256-byte runs (16 rows) of codes and
    // exponent bytes [w BN / 4, (w + 1) BN / 4) with its first BN / 16 lanes
    typedef W4Load<BN> L;
    const size_t kb = (size_t)(k / SK);
    uint8_t* b4 = (uint8_t*)s.b;
#pragma unroll
    for (int i = 0; i < L::loads; ++i)
      __builtin_amdgcn_global_load_lds((const void*)(src.w4[i] + kb * src.kstep * 16),
                                       (lds_void_t*)(b4 + (wave * L::loads + i) * 256), 4, 0, 0);
    if ((threadIdx.x & 63) < BN / 16)
      __builtin_amdgcn_global_load_lds((const void*)(src.we + kb * src.kstep), (lds_void_t*)(s.be + wave * (BN / 4)),
                                       4, 0, 0);
  } else {
#pragma unroll
    for (int i = 0; i < BN / (16 * NW); ++i) {
      const int r = (i * NW + wave) * 16;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(src.rw, (lds_void_t*)(s.b + r * SK), 16, src.w[i], 2 * k, 0, 0);
    }
  }
}

// One stage of MFMAs: NW waves in a 2 x (NW/2) arrangement, each
// accumulating a (BM/2) x (2BN/NW) sub-tile of MFMA 16x16x32 tiles.
template <int BM, int BN, int WQ, int NW = 4>
__device__ __forceinline__ void stage_mfma(const GemmStage<BM, BN, WQ>& s, MfmaTile<BM, BN, NW>& t, int wave) {
  constexpr int FM = BM / 32, FN = BN / (8 * NW), WCOL = 2 * BN / NW;
  const int lane = threadIdx.x & 63;
  const int wm = wave / (NW / 2), wn = wave % (NW / 2);
  const int r16 = lane & 15;
  const int pos = ((lane >> 4) ^ swz(r16)) * 8;   // fragment rows are r16 + 16 j
  u32x4 bfr[FN];
  if constexpr (WQ == WQ_FP8) {
    // fp8 rows of 32 B, unswizzled: a fragment's 16 rows are 512 contiguous bytes
    const uint8_t* b8 = (const uint8_t*)s.b;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const uint2 raw = *(const uint2*)(b8 + (wn * WCOL + j * 16 + r16) * SK + (lane >> 4) * 8);
      bfr[j] = __builtin_bit_cast(u32x4, fp8x8_to_bf16(raw));
    }
  } else if constexpr (WQ == WQ_MXFP4) {
    // E2M1 rows of 16 B: a fragment's 16 rows are 256 contiguous bytes; the
    // lane's 8 codes are 4 bytes, scaled by 2^(e - 127) (e >= 1; e = 0 only
    // in all-zero blocks, whose codes are zero)
    const uint8_t* b4 = (const uint8_t*)s.b;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int row = wn * WCOL + j * 16 + r16;
      const uint32_t raw = *(const uint32_t*)(b4 + row * 16 + (lane >> 4) * 4);
      const float sc = __uint_as_float((uint32_t)s.be[row] << 23);
      bfr[j] = __builtin_bit_cast(u32x4, fp4x8_to_bf16(raw, sc));
    }
  } else {
#pragma unroll
    for (int j = 0; j < FN; ++j) bfr[j] = *(const u32x4*)(&s.b[(wn * WCOL + j * 16 + r16) * SK + pos]);
  }
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int row = wm * (BM / 2) + i * 16 + r16;
    const bf16x8 ah = __builtin_bit_cast(bf16x8, *(const u32x4*)(&s.ah[row * SK + pos]));
    const bf16x8 al = __builtin_bit_cast(bf16x8, *(const u32x4*)(&s.al[row * SK + pos]));
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const bf16x8 bj = __builtin_bit_cast(bf16x8, bfr[j]);
      t.acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bj, t.acc[i][j], 0, 0, 0);
      t.acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bj, t.acc[i][j], 0, 0, 0);
    }
  }
}

// Main loop of one group of 4 waves (wave = 0..3 within the group) over the
// K range [k0, k0 + klen), klen a positive multiple of KALIGN.  The A rows
// are m0 + r, or gathered through arows (rows past nvalid repeat the first
// listed row; their results are discarded by the caller).  The four stages
// are separate LDS objects so the compiler can tell the loads into one stage
// from the reads of another.  All waves of the workgroup must run the same
// number of stages (the barriers are workgroup-wide).
// Weights: bf16 or fp8 rows of stride ldw, or (MXFP4) the stage-major block
// of ldw rows per 32-deep stage with the exponents wexp.
template <int BM, int BN, int WQ = WQ_NONE, int NW = 4>
__device__ __forceinline__ void mfma_mainloop(const bf16_t* __restrict__ A, int lda, size_t a_plane,
                                              const void* __restrict__ Wv, int ldw,
                                              const uint8_t* __restrict__ wexp, int k0,
                                              int klen, int m0, int n0, MfmaTile<BM, BN, NW>& t,
                                              GemmStage<BM, BN, WQ>& s0, GemmStage<BM, BN, WQ>& s1,
                                              GemmStage<BM, BN, WQ>& s2, GemmStage<BM, BN, WQ>& s3,
                                              int wave, const int32_t* __restrict__ arows = nullptr,
                                              int nvalid = 0) {
  // load instructions per thread per stage
  constexpr int LPS = 2 * (BM / (16 * NW)) +
                      (WQ == WQ_FP8 ? W8Load<BN>::loads
                                    : (WQ == WQ_MXFP4 ? W4Load<BN>::loads + 1 : BN / (16 * NW)));
  const int lane = threadIdx.x & 63;
  const int rsub = lane >> 2, chunk = (lane & 3) ^ swz(rsub);
  TileSrc<BM, BN, WQ, NW> src;
  // resources start at the tile's first row (gathered rows: at row 0, so a
  // plane's rows x lda x 2 bytes must stay below 4 GiB, checked on the host)
  const bf16_t* ab = A + (arows ? (size_t)0 : (size_t)m0 * lda) + k0;
  src.ra_h = __builtin_amdgcn_make_buffer_rsrc((void*)ab, 0, -1, BUF_DWORD3);
  src.ra_l = __builtin_amdgcn_make_buffer_rsrc((void*)(ab + a_plane), 0, -1, BUF_DWORD3);
#pragma unroll
  for (int i = 0; i < BM / (16 * NW); ++i) {
    const int r = (i * NW + wave) * 16 + rsub;
    const int grow = arows ? arows[r < nvalid ? r : 0] : r;
    src.a[i] = ((uint32_t)grow * (uint32_t)lda + chunk * 8) * 2u;
  }
  if constexpr (WQ == WQ_FP8) {
    typedef W8Load<BN> L;
    const uint8_t* W = (const uint8_t*)Wv;
    const int per_row = SK / L::bytes;       // lanes per 32-byte row
#pragma unroll
    for (int i = 0; i < L::loads; ++i) {
      const int r = (wave * L::loads + i) * L::rows + lane / per_row;
      src.w8[i] = W + (size_t)(n0 + r) * ldw + k0 + (lane % per_row) * L::bytes;
    }
  } else if constexpr (WQ == WQ_MXFP4) {
    typedef W4Load<BN> L;
    const size_t kb0 = (size_t)(k0 / SK);
    const uint8_t* W = (const uint8_t*)Wv + (kb0 * ldw + n0) * 16;
#pragma unroll
    for (int i = 0; i < L::loads; ++i) src.w4[i] = W + (wave * L::loads + i) * 256 + lane * 4;
    src.we = wexp + kb0 * ldw + n0 + wave * (BN / 4) + (lane < BN / 16 ? lane : 0) * 4;
    src.kstep = (size_t)ldw;
  } else {
    src.rw = __builtin_amdgcn_make_buffer_rsrc((void*)((const bf16_t*)Wv + (size_t)n0 * ldw + k0), 0, -1, BUF_DWORD3);
#pragma unroll
    for (int i = 0; i < BN / (16 * NW); ++i)
      src.w[i] = ((uint32_t)((i * NW + wave) * 16 + rsub) * (uint32_t)ldw + chunk * 8) * 2u;
  }
#pragma unroll
  for (int i = 0; i < BM / 32; ++i)
#pragma unroll
    for (int j = 0; j < BN / (8 * NW); ++j) t.acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int nk = klen / SK;     // multiple of 4, >= 4
  // no scalar load left in flight: the loop's LDS waits can then count the
  // fragment reads down instead of draining them
  __builtin_amdgcn_s_waitcnt(0xC07F);
  stage_issue<BM, BN, WQ, NW>(src, a_plane, 0, s0, wave);
  stage_issue<BM, BN, WQ, NW>(src, a_plane, SK, s1, wave);
  stage_issue<BM, BN, WQ, NW>(src, a_plane, 2 * SK, s2, wave);
  int kt = 0;
  // each step: own loads of stage kt done (the two younger stages may still
  // be in flight), barrier (everyone's loads done, everyone past stage kt-1),
  // refill the stage of kt-1 with kt+3, compute stage kt
#define BD_GEMM_STEP(CUR, NXT, KNEXT)                            \
  wait_vmcnt<2 * LPS>();                                         \
  __builtin_amdgcn_s_barrier();                                  \
  stage_issue<BM, BN, WQ, NW>(src, a_plane, (KNEXT) * SK, NXT, wave);    \
  stage_mfma<BM, BN, WQ, NW>(CUR, t, wave);
  for (; kt + 4 < nk; kt += 4) {
    BD_GEMM_STEP(s0, s3, kt + 3)
    BD_GEMM_STEP(s1, s0, kt + 4)
    BD_GEMM_STEP(s2, s1, kt + 5)
    BD_GEMM_STEP(s3, s2, kt + 6)
  }
#undef BD_GEMM_STEP
  // the last four stages (kt + 3 == nk - 1)
  wait_vmcnt<2 * LPS>();
  __builtin_amdgcn_s_barrier();
  stage_issue<BM, BN, WQ, NW>(src, a_plane, (kt + 3) * SK, s3, wave);
  stage_mfma<BM, BN, WQ, NW>(s0, t, wave);
  wait_vmcnt<2 * LPS>();
  __builtin_amdgcn_s_barrier();
  stage_mfma<BM, BN, WQ, NW>(s1, t, wave);
  wait_vmcnt<LPS>();
  __builtin_amdgcn_s_barrier();
  stage_mfma<BM, BN, WQ, NW>(s2, t, wave);
  wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  stage_mfma<BM, BN, WQ, NW>(s3, t, wave);
}

#define BD_GEMM_SMEM(BM, BN, WQ)                                                 \
  __shared__ __attribute__((aligned(1024))) GemmStage<BM, BN, WQ> gs0, gs1, gs2, gs3

// fp8 weights: multiply accumulator column n (of this wave's fragments) by
// the row scale sc[n] of the weight, a power of two.
template <int BM, int BN>
__device__ __forceinline__ void scale_columns(MfmaTile<BM, BN>& t, const float* __restrict__ sc, int n0,
                                              int wave) {
  const int lane = threadIdx.x & 63, wn = wave & 1;
#pragma unroll
  for (int j = 0; j < BN / 32; ++j) {
    const float f = sc[n0 + wn * (BN / 2) + j * 16 + (lane & 15)];
#pragma unroll
    for (int i = 0; i < BM / 32; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) t.acc[i][j][r] *= f;
  }
}

// GEMM, epilogue applied in registers.  Items (split z, column tile x, row
// tile y) are numbered z-major, then in bands of row tiles (band_tile): an
// XCD's concurrent workgroups share the A slices of a few row tiles and the
// W slices of a few column tiles of one split.  For
// EPI_ADD_F32 with a split workspace, the kernel picks S = resid_splits(M)
// K-splits on the device (zmax is the largest allowed); with S > 1 every
// split stores its raw partial tile to ws[split][row][col] (rows padded to
// whole tiles) and the next RMSNorm of the residual stream adds the partials
// in split order.
template <int BM, int BN, int EPI, int WQ, int NW = 4>
__global__ __launch_bounds__(64 * NW) void k_gemm_bf16(const bf16_t* __restrict__ A, int lda,
                                                   size_t a_plane, const void* __restrict__ W,
                                                   int ldw, int N, int K,
                                                   const int32_t* __restrict__ Mp,
                                                   void* __restrict__ out, int ldo, size_t out_plane,
                                                   float* __restrict__ ws, int zmax,
                                                   const void* __restrict__ waux) {
  constexpr int FM = BM / 32, FN = BN / (8 * NW), WCOL = 2 * BN / NW;
  const int M = *Mp;
  const int X = N / BN, Y = (M + BM - 1) / BM;
  int S = 1;
  if (EPI == EPI_ADD_F32 && ws) {
    ResidSplit r;
    r.nx = X; r.bm = BM; r.K = K; r.zmax = zmax;
    S = resid_splits(M, r);
  }
  const int items = X * Y * S;
  const int u = xcd_item(blockIdx.x, items);
  if (u >= items) return;
  const int z = u / (X * Y);
  int tx, ty;
  band_tile(u % (X * Y), X, Y, BAND_R, tx, ty);
  const int m0 = ty * BM, n0 = tx * BN;
  const int klen = K / S;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  BD_GEMM_SMEM(BM, BN, WQ);
  MfmaTile<BM, BN, NW> t;
  mfma_mainloop<BM, BN, WQ, NW>(A, lda, a_plane, W, WQ == WQ_MXFP4 ? N : ldw, (const uint8_t*)waux,
                                z * klen, klen, m0, n0, t, gs0, gs1, gs2, gs3, wave);
  if constexpr (WQ == WQ_FP8) scale_columns<BM, BN>(t, (const float*)waux, n0, wave);
  const int wm = wave / (NW / 2), wn = wave % (NW / 2);
  float* wz = (EPI == EPI_ADD_F32 && S > 1) ? ws + (size_t)z * ((M + BM - 1) / BM) * BM * N
                                            : nullptr;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + wm * (BM / 2) + i * 16 + (lane >> 4) * 4 + r;
      if (m >= M) continue;
      if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int j = 0; j < FN; j += 2) {
          const int pb = n0 + wn * WCOL + j * 16;        // packed column of the gate group
          const int col = (pb >> 5) * 16 + (lane & 15);  // output feature
          const float g = t.acc[i][j][r], u = t.acc[i][j + 1][r];
          store_pair((bf16_t*)out + (size_t)m * ldo + col, out_plane, silu(g) * u);
        }
      } else {
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int n = n0 + wn * WCOL + j * 16 + (lane & 15);
          const float v = t.acc[i][j][r];
          if (EPI == EPI_ADD_F32 && S > 1) wz[(size_t)m * N + n] = v;
          else if (EPI == EPI_ADD_F32) ((float*)out)[(size_t)m * ldo + n] += v;
          else ((float*)out)[(size_t)m * ldo + n] = v;
        }
      }
    }
  }
}

// QKV projection with RoPE and the K/V cache write in the epilogue (bf16).
// In the accumulator layout a lane holds rows mb + r (r < 4) of column n;
// the pair-interleaved weight puts the rotation partner of column n in
// column n ^ 1, i.e. lane ^ 1.  q and k: y(i) = x(i) cos - x(i + hd/2) sin,
// y(i + hd/2) = x(i + hd/2) cos + x(i) sin in fp64 with one rounding to
// fp32, stored at the original dimension; v: four consecutive rows of one
// sequence are four consecutive positions of one V^T tile row (one 8-byte store
// per plane).
__device__ __forceinline__ void store_pair4(bf16_t* p, size_t plane, const float v[4]) {
  bf16_t h[4], l[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    h[e] = f2bf(v[e]);
    l[e] = f2bf(v[e] - bf2f(h[e]));
  }
  *(uint2*)p = make_uint2((uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16));
  *(uint2*)(p + plane) =
      make_uint2((uint32_t)l[0] | ((uint32_t)l[1] << 16), (uint32_t)l[2] | ((uint32_t)l[3] << 16));
}

template <int BM, int BN, int WQ, int NW = 4>
__global__ __launch_bounds__(64 * NW) void k_gemm_qkv(const bf16_t* __restrict__ A, int lda,
                                                  size_t a_plane, const void* __restrict__ W,
                                                  int K, const int32_t* __restrict__ Mp, QkvEpi e,
                                                  const void* __restrict__ waux) {
  constexpr int FM = BM / 32, FN = BN / (8 * NW), WCOL = 2 * BN / NW;
  const int M = *Mp;
  const int X = (e.H + 2 * e.Hkv) * e.hd / BN, Y = (M + BM - 1) / BM;
  const int u = xcd_item(blockIdx.x, X * Y);
  if (u >= X * Y) return;
  int tx, ty;
  band_tile(u, X, Y, BAND_R, tx, ty);
  const int m0 = ty * BM, n0 = tx * BN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  BD_GEMM_SMEM(BM, BN, WQ);
  MfmaTile<BM, BN, NW> t;
  mfma_mainloop<BM, BN, WQ, NW>(A, lda, a_plane, W, WQ == WQ_MXFP4 ? X * BN : K, (const uint8_t*)waux, 0, K,
                                m0, n0, t, gs0, gs1, gs2, gs3, wave);
  if constexpr (WQ == WQ_FP8) scale_columns<BM, BN>(t, (const float*)waux, n0, wave);
  const int wm = wave / (NW / 2), wn = wave % (NW / 2);
  const int hd = e.hd, half = hd >> 1;
  const int qcols = e.H * hd, qkcols = (e.H + e.Hkv) * hd;
  bf16_t* Q = (bf16_t*)e.Q;
  bf16_t* Kc = (bf16_t*)e.kv.K;
  bf16_t* Vc = (bf16_t*)e.kv.V;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int mb = m0 + wm * (BM / 2) + i * 16 + (lane >> 4) * 4;   // the lane's first row
    int seq[4], pos[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const bool ok = mb + r < M;
      seq[r] = ok ? e.row_seq[mb + r] : 0;
      pos[r] = ok ? e.row_pos[mb + r] : 0;
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int n = n0 + wn * WCOL + j * 16 + (lane & 15);
      float v[4], pv[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        v[r] = t.acc[i][j][r];
        pv[r] = __shfl_xor(v[r], 1);
      }
      // a 16-column fragment lies inside one head, so the branch is uniform
      if (n < qkcols) {
        const int cp = n % hd, ip = cp >> 1;
        const bool odd = cp & 1;
        const int dim = odd ? ip + half : ip;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          if (mb + r >= M) continue;
          const double* cs = e.rope + ((size_t)pos[r] * half + ip) * 2;
          const double x1 = odd ? (double)pv[r] : (double)v[r];
          const double x2 = odd ? (double)v[r] : (double)pv[r];
          const float y = odd ? (float)(x2 * cs[0] + x1 * cs[1]) : (float)(x1 * cs[0] - x2 * cs[1]);
          if (n < qcols) {
            store_pair(Q + ((size_t)(mb + r) * e.H + n / hd) * hd + dim, e.q_plane, y);
          } else {
            const int kh = (n - qcols) / hd;
            store_pair(Kc + (((size_t)seq[r] * e.Hkv + kh) * e.kv.maxpos + pos[r]) * hd + dim,
                       e.kv.k_plane, y);
          }
        }
      } else {
        const int vn = n - qkcols, kh = vn / hd, dim = vn % hd;
        if (e.rows4 && mb + 3 < M) {
          store_pair4(Vc + ((size_t)seq[0] * e.Hkv + kh) * hd * e.kv.vstride + vt_off(pos[0], dim, hd),
                      e.kv.v_plane, v);
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (mb + r < M)
              store_pair(Vc + ((size_t)seq[r] * e.Hkv + kh) * hd * e.kv.vstride + vt_off(pos[r], dim, hd),
                         e.kv.v_plane, v[r]);
        }
      }
    }
  }
}

// Grouped GEMM over experts: tile ti covers rows [m0, m0 + 128) of expert
// tile_e[ti]; the expert's rows sit at [e_off[e], e_off[e] + e_cnt[e]) of the
// expert-sorted outputs.  The A rows are gathered through a_rows (token rows
// of the expert-sorted assignments) or, with a_rows == NULL, read from the
// expert-sorted layout itself.  W of expert e starts e * w_stride weight
// elements in (its codes, for quantized weights); fp8 row scales at
// waux + e * N, MXFP4 exponents at waux + e * w_stride / 32.
template <int EPI, int WQ, int NW = 4>
__global__ __launch_bounds__(64 * NW) void k_gemm_grouped(const bf16_t* __restrict__ A, int lda,
                                                      size_t a_plane, const void* __restrict__ W,
                                                      int ldw, int K, GroupTiles g,
                                                      void* __restrict__ out, int ldo,
                                                      size_t out_plane,
                                                      const void* __restrict__ waux, int N) {
  constexpr int BM = 128, BN = 128, FM = BM / 32, FN = BN / (8 * NW), WCOL = 2 * BN / NW;
  const int ti = blockIdx.y;
  if (ti >= *g.ntiles) return;
  const int e = g.tile_e[ti], m0 = g.tile_m0[ti];
  const int cnt = g.e_cnt[e], base = g.e_off[e];
  const int n0 = blockIdx.x * BN;
  BD_GEMM_SMEM(BM, BN, WQ);
  MfmaTile<BM, BN, NW> t;
  const size_t eoff = (size_t)e * g.w_stride;
  const void* We = WQ == WQ_NONE  ? (const void*)((const bf16_t*)W + eoff)
                   : WQ == WQ_FP8 ? (const void*)((const uint8_t*)W + eoff)
                                  : (const void*)((const uint8_t*)W + eoff / 2);
  const uint8_t* wexp = WQ == WQ_MXFP4 ? (const uint8_t*)waux + eoff / MX_BLOCK : nullptr;
  const int ldw_e = WQ == WQ_MXFP4 ? N : ldw;
  if (g.a_rows)
    mfma_mainloop<BM, BN, WQ, NW>(A, lda, a_plane, We, ldw_e, wexp, 0, K, 0, n0, t, gs0, gs1, gs2, gs3,
                              threadIdx.x >> 6, g.a_rows + base + m0, cnt - m0);
  else
    mfma_mainloop<BM, BN, WQ, NW>(A, lda, a_plane, We, ldw_e, wexp, 0, K, base + m0, n0, t, gs0, gs1, gs2, gs3,
                              threadIdx.x >> 6);
  if constexpr (WQ == WQ_FP8)
    scale_columns<BM, BN>(t, (const float*)waux + (size_t)e * N, n0, threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / (NW / 2), wn = wave % (NW / 2);
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
          const int pb = n0 + wn * WCOL + j * 16;
          const int col = (pb >> 5) * 16 + (lane & 15);
          store_pair((bf16_t*)out + orow * ldo + col, out_plane, silu(t.acc[i][j][r]) * t.acc[i][j + 1][r]);
        }
      } else {
#pragma unroll
        for (int j = 0; j < FN; ++j)
          ((float*)out)[orow * ldo + n0 + wn * WCOL + j * 16 + (lane & 15)] = t.acc[i][j][r];
      }
    }
  }
}

hipError_t launch_gemm_grouped(int epi, const void* A, int lda, size_t a_plane, const void* W,
                               int ldw, int N, int K, const GroupTiles& g, int max_tiles, void* out,
                               int ldo, size_t out_plane, WQuant wq, hipStream_t st) {
  if (N % 128 || K % KALIGN) return hipErrorInvalidValue;
  if ((wq.fmt != WQ_NONE) != (wq.aux != nullptr) || wq.fmt < WQ_NONE || wq.fmt > WQ_MXFP4)
    return hipErrorInvalidValue;
  dim3 grid(N / 128, max_tiles);
  const bf16_t* a = (const bf16_t*)A;
// waves per grouped tile: 8 (2 x 4 of 64 x 32) for the bf16 gate/up product
// (expert gate/up per MoE decode 366 -> 355 ms against 4 waves of 64 x 64),
// 4 for the down product (8 waves: 230 -> 234) and quantized weights
#define GROUPED_NW(EPI_, WQ_) ((EPI_) == EPI_SWIGLU && (WQ_) == WQ_NONE ? 8 : 4)
#define BD_GROUPED(EPI_, WQ_, OP_) \
  k_gemm_grouped<EPI_, WQ_, GROUPED_NW(EPI_, WQ_)><<<grid, 64 * GROUPED_NW(EPI_, WQ_), 0, st>>>(a, lda, a_plane, W, \
                                                                                              ldw, K, g, out, ldo, OP_, \
                                                                                              wq.aux, N)
  if (epi == EPI_SWIGLU) {
    if (wq.fmt == WQ_FP8) BD_GROUPED(EPI_SWIGLU, WQ_FP8, out_plane);
    else if (wq.fmt == WQ_MXFP4) BD_GROUPED(EPI_SWIGLU, WQ_MXFP4, out_plane);
    else BD_GROUPED(EPI_SWIGLU, WQ_NONE, out_plane);
  } else {
    if (wq.fmt == WQ_FP8) BD_GROUPED(EPI_STORE_F32, WQ_FP8, 0);
    else if (wq.fmt == WQ_MXFP4) BD_GROUPED(EPI_STORE_F32, WQ_MXFP4, 0);
    else BD_GROUPED(EPI_STORE_F32, WQ_NONE, 0);
  }
#undef BD_GROUPED
#undef GROUPED_NW
  return hipGetLastError();
}

// Fused LM head: for its TBN vocabulary columns the workgroup reduces each row
// to (max z, sum exp(z - max), lowest argmax) and writes one partial per
// (column tile, row); logits never leave registers.  Tiles of 128 x 256
// with 8 waves of 64 x 64 (the gate/up tile) where the LM rows reach 2048,
// else 128 x 128 with 4 waves of 64 x 64: on the multi-block decode's
// 3072-row capacity the LM head went from 1065 to 772 us per launch.
template <int TBN, int NW>
__global__ __launch_bounds__(64 * NW) void k_lm_head_bf16(const bf16_t* __restrict__ A, int d,
                                                      size_t a_plane,
                                                      const bf16_t* __restrict__ W, int V, int mask_id,
                                                      float scale, const int32_t* __restrict__ Mp,
                                                      int rows_cap, float* __restrict__ pmax,
                                                      float* __restrict__ psum,
                                                      int32_t* __restrict__ parg) {
  constexpr int TBM = 128, FN = TBN / (8 * NW), WCOL = 2 * TBN / NW, NP = NW / 2;
  const int M = *Mp;
  // items in bands of row tiles (band_tile): an XCD's concurrent workgroups
  // share a few row tiles of the operand and a few vocabulary tiles of the head
  const int X = V / TBN, Y = (M + TBM - 1) / TBM;
  const int u = xcd_item(blockIdx.x, X * Y);
  if (u >= X * Y) return;
  int vt, ty;
  band_tile(u, X, Y, BAND_R, vt, ty);
  const int m0 = ty * TBM, n0 = vt * TBN;
  BD_GEMM_SMEM(TBM, TBN, WQ_NONE);
  // per-row partials of the NP column groups of waves
  __shared__ float red_m[NP][TBM], red_s[NP][TBM];
  __shared__ int32_t red_a[NP][TBM];
  MfmaTile<TBM, TBN, NW> t;
  mfma_mainloop<TBM, TBN, WQ_NONE, NW>(A, d, a_plane, W, d, nullptr, 0, d, m0, n0, t, gs0, gs1, gs2, gs3,
                                       threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / NP, wn = wave % NP;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float v[FN];
      float mx = -INFINITY;
      int arg = 0x7fffffff;
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int n = n0 + wn * WCOL + j * 16 + (lane & 15);
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
      for (int j = 0; j < FN; ++j) s += expf(v[j] - mx);
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
      // column groups in order: the first group holding the maximum gives
      // the (lowest) argmax
      float mm = red_m[0][rl];
      int a = red_a[0][rl];
#pragma unroll
      for (int p = 1; p < NP; ++p)
        if (red_m[p][rl] > mm) { mm = red_m[p][rl]; a = red_a[p][rl]; }
      float s = 0.f;
#pragma unroll
      for (int p = 0; p < NP; ++p) s += red_s[p][rl] * expf(red_m[p][rl] - mm);
      const size_t o = (size_t)vt * rows_cap + m;
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

template <int BM, int BN, int WQ, int NW = 4>
static void launch_bf16_cfg(int epi, dim3 grid, const bf16_t* a, int lda, size_t ap, const void* w,
                            int ldw, int N, int K, const int32_t* M_dev, void* o, int ldo, size_t op,
                            float* ws, int zmax, const void* waux, hipStream_t st) {
  switch (epi) {
    case EPI_ADD_F32:
      k_gemm_bf16<BM, BN, EPI_ADD_F32, WQ, NW><<<grid, 64 * NW, 0, st>>>(a, lda, ap, w, ldw, N, K, M_dev, o, ldo, op, ws,
                                                                 zmax, waux);
      break;
    case EPI_SWIGLU:
      k_gemm_bf16<BM, BN, EPI_SWIGLU, WQ, NW><<<grid, 64 * NW, 0, st>>>(a, lda, ap, w, ldw, N, K, M_dev, o, ldo, op,
                                                                nullptr, 1, waux);
      break;
    default:
      k_gemm_bf16<BM, BN, EPI_STORE_F32, WQ, NW><<<grid, 64 * NW, 0, st>>>(a, lda, ap, w, ldw, N, K, M_dev, o, ldo, op,
                                                                   nullptr, 1, waux);
      break;
  }
}

// Tile choice: 128x256 (8 waves of 64 x 64, two per SIMD; 128 KB of LDS) over
// windows of at least 2048 rows for wide plain products (N >= 8192) and
// residual ones with K >= 2048, when the caller allows it (bf16 weights and a
// kernel instantiated for it): on
// 3328-row products it ran gate/up (N 16384) in 494 us against 550 and down
// (N 2048, K 8192) in 259 against 291.  With 8 waves per tile the shallower
// O projection (N 2048, K 2048) gains too, even where few rows are live: per
// decode 256 -> 193 ms on the multi-block window, 90 -> 71 on the MoE window
// (about 2300 live rows of 4096), 56 -> 39 on the long-prefix window.
// Otherwise 128x128 when that tiling gives enough workgroups over the row
// capacity (the 64x64 tile runs out of LDS bandwidth on large products),
// else 64x64.  Enough: 1024 for plain products (below that the 128x128 grid
// leaves part of the chip idle for a round: the gate/up product of the dense
// decode, 512 workgroups over its 1024-row capacity, runs 6% faster in
// 64x64 tiles), 512 for residual projections, whose split-K partials grow
// with the tile count (the multi-block O projection ran 18% slower in 64x64
// tiles).  Plain products over windows of at most 1024 rows take 64x128
// instead of 64x64 (bf16 weights): half the re-reads of the activation per
// column tile, two workgroups per CU; the dense decode's gate/up product
// went from 27.3 to 24.0 us per launch, while the MoE window's (4096 rows)
// shared-expert products ran 1.5-3% slower in it.  zmax: the largest
// residual split (1 = none).
GemmPlan plan_gemm(bool is_bf16, int N, int K, int rows_cap, bool resid, bool wide_ok) {
  if (!is_bf16) return GemmPlan{64, 64, 1};
  if (wide_ok && N % 256 == 0 && rows_cap >= 2048 && (N >= 8192 || (resid && K >= 2048)))
    return GemmPlan{128, 256, 1};
  if (N % 128 == 0 && (N / 128) * cdiv(rows_cap, 128) >= (resid ? 512 : 1024)) return GemmPlan{128, 128, 1};
  if (wide_ok && !resid && N % 128 == 0 && rows_cap <= 1024) return GemmPlan{64, 128, 1};
  return GemmPlan{64, 64, 1};
}

hipError_t launch_gemm_planned(const GemmPlan& p, int epi, const void* A, int lda, size_t a_plane,
                               const void* W, int ldw, int N, int K, const int32_t* M_dev,
                               int rows_cap, void* out, int ldo, size_t out_plane, float* ws,
                               hipStream_t st, WQuant wq) {
  const bool big = p.bm == 128 && p.bn == 128, small = p.bm == 64 && p.bn == 64;
  const bool wide = p.bm == 128 && p.bn == 256, mid = p.bm == 64 && p.bn == 128;
  if ((!big && !small && !wide && !mid) || p.zmax < 1 || p.zmax > 8) return hipErrorInvalidValue;
  if ((wq.fmt != WQ_NONE) != (wq.aux != nullptr) || wq.fmt < WQ_NONE || wq.fmt > WQ_MXFP4)
    return hipErrorInvalidValue;
  if ((wide || mid) && wq.fmt != WQ_NONE) return hipErrorInvalidValue;   // no quantized variants
  if (mid && p.zmax != 1) return hipErrorInvalidValue;
  if (N % p.bn || K % KALIGN) return hipErrorInvalidValue;
  if (p.zmax > 1 && (epi != EPI_ADD_F32 || !ws)) return hipErrorInvalidValue;
  // 1-D grid: every (split, column tile, row tile) of the row capacity, + 7
  // (see xcd_item)
  dim3 grid((N / p.bn) * cdiv(rows_cap, p.bm) * p.zmax + 7);
  const bf16_t* a = (const bf16_t*)A;
#define BD_CFG(BM_, BN_, WQ_) \
  launch_bf16_cfg<BM_, BN_, WQ_>(epi, grid, a, lda, a_plane, W, ldw, N, K, M_dev, out, ldo, out_plane, ws, p.zmax, \
                                 wq.aux, st)
  if (wq.fmt == WQ_FP8) {
    if (big) BD_CFG(128, 128, WQ_FP8); else BD_CFG(64, 64, WQ_FP8);
  } else if (wq.fmt == WQ_MXFP4) {
    if (big) BD_CFG(128, 128, WQ_MXFP4); else BD_CFG(64, 64, WQ_MXFP4);
  } else {
    if (wide) launch_bf16_cfg<128, 256, WQ_NONE, 8>(epi, grid, a, lda, a_plane, W, ldw, N, K, M_dev, out, ldo,
                                                     out_plane, ws, p.zmax, nullptr, st);
    else if (big) BD_CFG(128, 128, WQ_NONE);
    else if (mid) BD_CFG(64, 128, WQ_NONE);
    else BD_CFG(64, 64, WQ_NONE);
  }
#undef BD_CFG
  return hipGetLastError();
}

size_t resid_extent(int M, int N, const ResidSplit& r) {
  if (M < 1) return 0;
  const int S = resid_splits(M, r);
  return S > 1 ? (size_t)S * (size_t)cdiv(M, r.bm) * r.bm * N : 0;
}

size_t resid_extent_max(int rows_cap, int N, const ResidSplit& r) {
  // S and the slab height depend on M only through its row-tile count
  size_t mx = 0;
  for (int y = 1; y <= cdiv(rows_cap, r.bm); ++y) {
    const size_t e = resid_extent(y * r.bm < rows_cap ? y * r.bm : rows_cap, N, r);
    if (e > mx) mx = e;
  }
  return mx;
}

GemmPlan plan_resid(int N, int K, int rows_cap, bool wide_ok) {
  // deep products (K >= 4096) take 128-row tiles: with K split, their A and
  // W re-reads halve against 64x64 at the same parallelism
  GemmPlan p = plan_gemm(true, N, K, rows_cap, true, wide_ok);
  if (K >= 4096 && N % 128 == 0 && p.bm != 128) p = GemmPlan{128, 128, 1};
  p.zmax = 8;
  return p;
}

hipError_t launch_gemm_resid(bool is_bf16, const void* A, int lda, size_t a_plane, const void* W,
                             int ldw, int N, int K, const int32_t* M_dev, int rows_cap, float* X,
                             int ldx, float* ws, size_t ws_floats, ResidSplit* fold, hipStream_t st,
                             WQuant wq) {
  fold->ws = nullptr;
  if (!is_bf16 || !ws)
    return launch_gemm(EPI_ADD_F32, is_bf16, A, lda, a_plane, W, ldw, N, K, M_dev, rows_cap, X, ldx, 0, st,
                       wq);
  const GemmPlan p = plan_resid(N, K, rows_cap, wq.fmt == WQ_NONE);
  ResidSplit r{};
  r.nx = N / p.bn;
  r.bm = p.bm;
  r.K = K;
  r.zmax = p.zmax;
  if (resid_extent_max(rows_cap, N, r) > ws_floats) return hipErrorInvalidValue;
  hipError_t e = launch_gemm_planned(p, EPI_ADD_F32, A, lda, a_plane, W, ldw, N, K, M_dev, rows_cap,
                                     X, ldx, 0, ws, st, wq);
  if (e != hipSuccess) return e;
  r.ws = ws;
  r.Mp = M_dev;
  *fold = r;
  return hipSuccess;
}

hipError_t launch_gemm_qkv(const void* A, int lda, size_t a_plane, const void* W, int K,
                           const int32_t* M_dev, int rows_cap, const QkvEpi& e, hipStream_t st,
                           WQuant wq) {
  const int N = (e.H + 2 * e.Hkv) * e.hd;
  if (e.hd % 16 || e.kv.vstride % 64 || K % KALIGN) return hipErrorInvalidValue;
  if ((wq.fmt != WQ_NONE) != (wq.aux != nullptr) || wq.fmt < WQ_NONE || wq.fmt > WQ_MXFP4)
    return hipErrorInvalidValue;
  // bf16 weights where the product would fill at least 512 tiles of 128 x 256
  // over the row capacity (the 6144-row multi-block window of a 3072-wide
  // QKV): 128x128 tiles with 8 waves of 64 x 32.  Per
  // decode, QKV took 428 ms in 4-wave 128x128 tiles, 383 in 8-wave 128x256
  // tiles (312 tiles for 256 CUs: a nearly empty second round) and 335 in
  // 8-wave 128x128 tiles (624 tiles, three half-length rounds).  The MoE
  // (4096-row) and long-prefix (2048-row) windows, whose live rows fall well
  // below the capacity, keep the 4-wave tiling: 8-wave tiles there ran 13%
  // slower and no faster.
  GemmPlan p = plan_gemm(true, N, K, rows_cap, false, false);
  const bool eight = wq.fmt == WQ_NONE && N % 256 == 0 && (N / 256) * cdiv(rows_cap, 128) >= 512;
  if (eight) p = GemmPlan{128, 128, 1};
  if (N % p.bn) return hipErrorInvalidValue;
  dim3 grid((N / p.bn) * cdiv(rows_cap, p.bm) + 7);
  const bf16_t* a = (const bf16_t*)A;
#define BD_QKV(BM_, WQ_) k_gemm_qkv<BM_, BM_, WQ_><<<grid, 256, 0, st>>>(a, lda, a_plane, W, K, M_dev, e, wq.aux)
  if (wq.fmt == WQ_FP8) {
    if (p.bm == 128) BD_QKV(128, WQ_FP8); else BD_QKV(64, WQ_FP8);
  } else if (wq.fmt == WQ_MXFP4) {
    if (p.bm == 128) BD_QKV(128, WQ_MXFP4); else BD_QKV(64, WQ_MXFP4);
  } else if (eight) {
    k_gemm_qkv<128, 128, WQ_NONE, 8><<<grid, 512, 0, st>>>(a, lda, a_plane, W, K, M_dev, e, nullptr);
  } else {
    if (p.bm == 128) BD_QKV(128, WQ_NONE); else BD_QKV(64, WQ_NONE);
  }
#undef BD_QKV
  return hipGetLastError();
}

hipError_t launch_gemm(int epi, bool is_bf16, const void* A, int lda, size_t a_plane, const void* W,
                       int ldw, int N, int K, const int32_t* M_dev, int rows_cap, void* out, int ldo,
                       size_t out_plane, hipStream_t st, WQuant wq) {
  if (is_bf16)
    return launch_gemm_planned(plan_gemm(true, N, K, rows_cap, false, wq.fmt == WQ_NONE), epi, A, lda, a_plane,
                               W, ldw, N, K, M_dev, rows_cap, out, ldo, out_plane, nullptr, st, wq);
  if (wq.fmt != WQ_NONE) return hipErrorInvalidValue;
  if (N % SBN || K % SBK) return hipErrorInvalidValue;
  dim3 grid(N / SBN, cdiv(rows_cap, SBM));
  const float* a = (const float*)A;
  const float* w = (const float*)W;
  switch (epi) {
    case EPI_ADD_F32: k_gemm_f32<EPI_ADD_F32><<<grid, 256, 0, st>>>(a, lda, w, ldw, N, K, M_dev, out, ldo); break;
    case EPI_SWIGLU: k_gemm_f32<EPI_SWIGLU><<<grid, 256, 0, st>>>(a, lda, w, ldw, N, K, M_dev, out, ldo); break;
    default: k_gemm_f32<EPI_STORE_F32><<<grid, 256, 0, st>>>(a, lda, w, ldw, N, K, M_dev, out, ldo); break;
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
    if (V % 128 || d % KALIGN) return hipErrorInvalidValue;
    const bool wide = V % 256 == 0 && rows_cap >= 2048;
    ntiles = V / (wide ? 256 : 128);
    dim3 grid(ntiles * cdiv(rows_cap, 128) + 7);
    if (wide)
      k_lm_head_bf16<256, 8><<<grid, 512, 0, st>>>((const bf16_t*)A, d, a_plane, (const bf16_t*)W, V, mask_id,
                                                   scale, M_dev, rows_cap, part_max, part_sum, part_arg);
    else
      k_lm_head_bf16<128, 4><<<grid, 256, 0, st>>>((const bf16_t*)A, d, a_plane, (const bf16_t*)W, V, mask_id,
                                                   scale, M_dev, rows_cap, part_max, part_sum, part_arg);
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
                             logits, V, 0, st);
  if (e != hipSuccess) return e;
  k_logits_post<<<dim3(cdiv(V, 256 * 8), rows_cap), 256, 0, st>>>(logits, V, mask_id, scale, M_dev);
  return hipGetLastError();
}

}  // namespace bd
