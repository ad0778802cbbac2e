// Block-causal attention over the KV cache (paper §2.1): a query at absolute
// position p attends to every key j with j / B <= p / B, i.e. the cached
// prefix, every earlier block and its own block (bidirectionally).  Window
// K/V have already been written into the cache at their absolute positions,
// so one key range [0, end of the query's block) covers prefix and window.
//
// bf16 kernel (Q, K and V are bf16 hi/lo pairs in two planes; V is kept
// transposed in the cache, in tiles of 64 keys [dim][64 slots], the keys of
// each 32-key group in the slot order of vt_slot): one workgroup =
// 16 NW queries of one (sequence, kv head) -- window rows x the q-heads that
// share the kv head -- as NW wave64s x 16 queries (NW = 2 when a window
// holds at most 32 such queries, 8 for 512 or more over long key ranges,
// else 4); a wave with no query of its own
// only helps stage the tiles.  Key tiles of 64
// positions stream from HBM through LDS with 16-byte coalesced loads (K rows
// and V^T tile rows, each tile a contiguous block), and the wave computes
// S^T = K Q^T and O^T += V^T P^T with MFMA 16x16x32 bf16 (three products
// hi.hi + hi.lo + lo.hi per pair of operands; the output leaves as the hi/lo
// pair of the next matmul operand), so each lane owns one query column: the
// online-softmax state and the O rescale stay in the lane, and P^T is fed to
// the second MFMA straight from the score registers (the two products use
// the same permutation of the key index).  The block mask is applied in
// registers, only on tiles that reach the query's block.
#include "bd_internal.h"

#include <math.h>

namespace bd {

__device__ __forceinline__ float bf2f_a(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }
__device__ __forceinline__ bf16_t f2bf_a(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

constexpr int AK = 64;    // keys per tile
// Fourth word of a raw buffer resource (gfx9 family): 32-bit data format (a
// zero format reads zeros), no index stride.
constexpr int ATT_BUF_DWORD3 = 0x00020000;

typedef __bf16 bf16x2_a __attribute__((ext_vector_type(2)));
typedef float floatx2_a __attribute__((ext_vector_type(2)));

// (x0, x1) -> the hi bf16 pair (round to nearest even, one v_cvt_pk_bf16_f32)
// in hi and the lo pair, the rounded remainders x - hi (exact in fp32), in lo
__device__ __forceinline__ void split_pair2(float x0, float x1, uint32_t& hi, uint32_t& lo) {
  hi = __builtin_bit_cast(uint32_t, __builtin_convertvector((floatx2_a){x0, x1}, bf16x2_a));
  const float h0 = __uint_as_float(hi << 16), h1 = __uint_as_float(hi & 0xFFFF0000u);
  lo = __builtin_bit_cast(uint32_t, __builtin_convertvector((floatx2_a){x0 - h0, x1 - h1}, bf16x2_a));
}

template <int HD, int NW>
__global__ __launch_bounds__(64 * NW) void k_attn_bf16(const bf16_t* __restrict__ Q, size_t q_plane,
                                                   const bf16_t* __restrict__ Kc, size_t k_plane,
                                                   const bf16_t* __restrict__ Vt, size_t v_plane,
                                                   int vstride, bf16_t* __restrict__ O,
                                                   size_t o_plane,
                                                   const int32_t* __restrict__ seq_row_start,
                                                   const int32_t* __restrict__ seq_win_len,
                                                   const int32_t* __restrict__ seq_win_start, int H,
                                                   int Hkv, int maxpos, int B, float scale_log2,
                                                   int kv_splits, float* __restrict__ ws_o,
                                                   float* __restrict__ ws_ml, int rows_cap,
                                                   int b, int nqt) {
  constexpr int KP = HD + 8;        // padded K row (elements)
  constexpr int VP = AK + 8;        // padded transposed-V row
  constexpr int CH = AK * HD / 8;   // 16-byte chunks per K (or V) tile and plane
  constexpr int NT = 64 * NW;       // threads
  constexpr int AQ = 16 * NW;       // queries per workgroup
  constexpr int NCH = CH / NT;      // chunks per thread
  __shared__ __attribute__((aligned(16))) bf16_t sKh[AK * KP];
  __shared__ __attribute__((aligned(16))) bf16_t sKl[AK * KP];
  __shared__ __attribute__((aligned(16))) bf16_t sVh[HD * VP];
  __shared__ __attribute__((aligned(16))) bf16_t sVl[HD * VP];

  // The queries of one (sequence s, kv head kv) are numbered qi = r * G + j
  // for window row r and q-head kv * G + j (G = H / Hkv heads share the kv
  // head); a workgroup takes AQ consecutive qi, so every K/V tile it stages
  // serves all G heads of the rows it covers.
  // Items u = ((s * Hkv + kv) * kv_splits + split) * nqt + qt: the nqt query
  // tiles that read the same keys are neighbours, so they share one XCD's L2.
  const int G = H / Hkv;
  const int items = b * Hkv * kv_splits * nqt;
  const int u = xcd_item(blockIdx.x, items);
  if (u >= items) return;
  const int qt = u % nqt, split = (u / nqt) % kv_splits;
  const int kv = (u / (nqt * kv_splits)) % Hkv, s = u / (nqt * kv_splits * Hkv);
  const int W = seq_win_len[s];
  const int QG = G * W;
  if (qt * AQ >= QG) return;
  const int row_start = seq_row_start[s], win_start = seq_win_start[s];
  const int qlast = min(qt * AQ + AQ, QG) - 1;
  const int kend = ((win_start + qlast / G) / B + 1) * B;   // keys [0, kend): the last row's bound
  // this split's key tiles: a contiguous, tile-aligned share of [0, kend)
  const int ntiles_all = (kend + AK - 1) / AK;
  const int per = (ntiles_all + kv_splits - 1) / kv_splits;
  const int t_lo = split * per, t_hi = min(ntiles_all, t_lo + per);
  const bf16_t* Kp = Kc + ((size_t)s * Hkv + kv) * (size_t)maxpos * HD;
  const bf16_t* Vp = Vt + ((size_t)s * Hkv + kv) * (size_t)HD * vstride;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  const int qi = qt * AQ + wave * 16 + c;                    // this lane's query
  const bool qvalid = qi < QG;
  const bool wave_on = qt * AQ + wave * 16 < QG;             // the wave holds a query
  const int qrow = row_start + (qvalid ? qi / G : 0);        // its row in the step
  const int h = kv * G + (qvalid ? qi % G : 0);              // its q-head
  const int qend = ((win_start + (qvalid ? qi / G : 0)) / B + 1) * B;   // its key bound
  // the wave's smallest key bound (query index and bound rise together) and
  // whether every lane holds a query: tiles below the bound skip the mask
  const int q0w = qt * AQ + wave * 16;
  const int qend_w = ((win_start + min(q0w, QG - 1) / G) / B + 1) * B;
  const bool full_w = q0w + 16 <= QG;

  // Q^T fragments (B operand of S^T = K Q^T): dims [32 kc + 8 g, +8) of query c,
  // hi and lo halves.
  bf16x8 qh[HD / 32], ql[HD / 32];
#pragma unroll
  for (int kc = 0; kc < HD / 32; ++kc) {
    if (qvalid) {
      const bf16_t* qp = Q + ((size_t)qrow * H + h) * HD + kc * 32 + g * 8;
      qh[kc] = __builtin_bit_cast(bf16x8, *(const u32x4*)qp);
      ql[kc] = __builtin_bit_cast(bf16x8, *(const u32x4*)(qp + q_plane));
    } else {
      qh[kc] = bf16x8{};
      ql[kc] = bf16x8{};
    }
  }
  floatx4 oacc[HD / 16];
#pragma unroll
  for (int t = 0; t < HD / 16; ++t) oacc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_part = 0.f;

  // register prefetch of the next K/V tile (both planes) overlaps the loads
  // with the MFMAs of the current tile.  K: chunk ci = (key, 8 dims), read
  // through a buffer resource that starts at the tile's first key and ends
  // at key kend, so keys >= kend (past the slice's written rows, possibly
  // past the slice) read zeros, finite scores that every query masks.  V^T:
  // chunk ci = (dim, 8 keys) of the tile's [HD][64] block; a tile never
  // reaches past vstride and the keys past kend there are finite cache
  // contents that meet zero probabilities.  The lanes' byte offsets inside a
  // tile do not change from tile to tile.
  u32x4 pkh[NCH], pkl[NCH], pvh[NCH], pvl[NCH];
  uint32_t kof[NCH], vof[NCH];
#pragma unroll
  for (int it = 0; it < NCH; ++it) {
    const int ci = tid + NT * it;
    kof[it] = (uint32_t)((ci / (HD / 8)) * HD + (ci % (HD / 8)) * 8) * 2u;
    vof[it] = (uint32_t)((ci / (AK / 8)) * AK + (ci % (AK / 8)) * 8) * 2u;
  }
#define BD_FETCH(K0)                                                                              \
  do {                                                                                            \
    const bf16_t* kb_ = Kp + (size_t)(K0) * HD;                                                   \
    const bf16_t* vb_ = Vp + (size_t)(K0) * HD;                                                   \
    const int nrec_ = max(kend - (K0), 0) * HD * 2;                                               \
    const __amdgpu_buffer_rsrc_t rkh_ = __builtin_amdgcn_make_buffer_rsrc((void*)kb_, 0, nrec_, ATT_BUF_DWORD3); \
    const __amdgpu_buffer_rsrc_t rkl_ =                                                           \
        __builtin_amdgcn_make_buffer_rsrc((void*)(kb_ + k_plane), 0, nrec_, ATT_BUF_DWORD3);      \
    const __amdgpu_buffer_rsrc_t rvh_ = __builtin_amdgcn_make_buffer_rsrc((void*)vb_, 0, AK * HD * 2, ATT_BUF_DWORD3); \
    const __amdgpu_buffer_rsrc_t rvl_ =                                                           \
        __builtin_amdgcn_make_buffer_rsrc((void*)(vb_ + v_plane), 0, AK * HD * 2, ATT_BUF_DWORD3); \
    _Pragma("unroll") for (int it = 0; it < NCH; ++it) {                                          \
      pkh[it] = __builtin_amdgcn_raw_buffer_load_b128(rkh_, kof[it], 0, 0);                       \
      pkl[it] = __builtin_amdgcn_raw_buffer_load_b128(rkl_, kof[it], 0, 0);                       \
      pvh[it] = __builtin_amdgcn_raw_buffer_load_b128(rvh_, vof[it], 0, 0);                       \
      pvl[it] = __builtin_amdgcn_raw_buffer_load_b128(rvl_, vof[it], 0, 0);                       \
    }                                                                                             \
  } while (0)
  if (t_lo < t_hi) BD_FETCH(t_lo * AK);
  for (int kt = t_lo; kt < t_hi; ++kt) {
    const int k0 = kt * AK;
    // stage K (row-major) and V^T
#pragma unroll
    for (int it = 0; it < NCH; ++it) {
      const int ci = tid + NT * it;
      const int key = ci / (HD / 8), dc = (ci % (HD / 8)) * 8;
      *(u32x4*)(sKh + key * KP + dc) = pkh[it];
      *(u32x4*)(sKl + key * KP + dc) = pkl[it];
      const int dim = ci / (AK / 8), kc8 = (ci % (AK / 8)) * 8;
      *(u32x4*)(sVh + dim * VP + kc8) = pvh[it];
      *(u32x4*)(sVl + dim * VP + kc8) = pvl[it];
    }
    __syncthreads();
    if (kt + 1 < t_hi) BD_FETCH(k0 + AK);
    if (wave_on) {

    // S^T sub-tiles (keys st*16 + 4g + r, query c): Kh.Qh + Kh.Ql + Kl.Qh
    float sv[4][4];
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      floatx4 a = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kc = 0; kc < HD / 32; ++kc) {
        const int off = (st * 16 + c) * KP + kc * 32 + g * 8;
        const bf16x8 kh = __builtin_bit_cast(bf16x8, *(const u32x4*)(sKh + off));
        const bf16x8 kl = __builtin_bit_cast(bf16x8, *(const u32x4*)(sKl + off));
        a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kh, qh[kc], a, 0, 0, 0);
        a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kh, ql[kc], a, 0, 0, 0);
        a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kl, qh[kc], a, 0, 0, 0);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) sv[st][r] = a[r];
    }
    // In this lane, score (st, r) belongs to key k0 + st*16 + 4g + r of query c.
    // Scores stay unscaled until the exponent: the max of the raw scores
    // times the (positive) scale is the max of the scaled ones.  The mask
    // branch is wave-uniform.
    if (k0 + AK > qend_w || !full_w) {
#pragma unroll
      for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = k0 + st * 16 + 4 * g + r;
          if (!qvalid || key >= qend) sv[st][r] = -INFINITY;
        }
    }
    float tmax = -INFINITY;
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int r = 0; r < 4; ++r) tmax = fmaxf(tmax, sv[st][r]);
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    const float m_new = fmaxf(m_run, tmax * scale_log2);
    const float m_ref = (m_new == -INFINITY) ? 0.f : m_new;
    // rescale only when some lane's running max moved (alpha = 1 elsewhere);
    // v_exp_f32 is exp2 without the denormal-range scaling: terms below
    // 2^-126 of the row max contribute nothing at fp32 precision anyway
    if (__any(m_new != m_run)) {
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_ref);
      l_part *= alpha;
#pragma unroll
      for (int t = 0; t < HD / 16; ++t) oacc[t] *= alpha;
    }
    m_run = m_new;
    // P^T as a hi/lo bf16 pair: keys 4g + r of sub-tile st take slots
    // (st & 1) * 4 + r of chunk st >> 1, two slots per 32-bit word
    uint32_t hw[4][2], lw[4][2];
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int r2 = 0; r2 < 2; ++r2) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(sv[st][2 * r2], scale_log2, -m_ref));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(sv[st][2 * r2 + 1], scale_log2, -m_ref));
        l_part += p0;
        l_part += p1;
        split_pair2(p0, p1, hw[st][r2], lw[st][r2]);
      }
    bf16x8 ph[2], pl[2];
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      ph[kc] = __builtin_bit_cast(bf16x8, u32x4{hw[2 * kc][0], hw[2 * kc][1], hw[2 * kc + 1][0], hw[2 * kc + 1][1]});
      pl[kc] = __builtin_bit_cast(bf16x8, u32x4{lw[2 * kc][0], lw[2 * kc][1], lw[2 * kc + 1][0], lw[2 * kc + 1][1]});
    }
    // O^T += V^T P^T over 2 chunks of 32 keys; k-slot 8g+r <-> key 32kc+4g+r,
    // k-slot 8g+4+r <-> key 32kc+16+4g+r (same permutation as the scores),
    // which the V^T slot order (vt_slot) stores as slots 32kc+8g..+7: one
    // 16-byte read per plane.  Vh.Ph + Vh.Pl + Vl.Ph
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
#pragma unroll
      for (int t = 0; t < HD / 16; ++t) {
        const int off = (t * 16 + c) * VP + kc * 32 + 8 * g;
        const bf16x8 vh = __builtin_bit_cast(bf16x8, *(const u32x4*)(sVh + off));
        const bf16x8 vl = __builtin_bit_cast(bf16x8, *(const u32x4*)(sVl + off));
        oacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vh, ph[kc], oacc[t], 0, 0, 0);
        oacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vh, pl[kc], oacc[t], 0, 0, 0);
        oacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vl, ph[kc], oacc[t], 0, 0, 0);
      }
    }
    }  // wave_on
    __syncthreads();
  }
#undef BD_FETCH
  float l = l_part;
  l += __shfl_xor(l, 16);
  l += __shfl_xor(l, 32);
  if (!qvalid) return;
  if (kv_splits == 1) {
    const float inv = 1.0f / l;
    bf16_t* orow = O + (size_t)qrow * H * HD + h * HD;
#pragma unroll
    for (int t = 0; t < HD / 16; ++t) {
      // O^T tile t: lane holds dims t*16 + 4g + r of query c; stored as the
      // bf16 pair (hi, lo) of the O-projection operand
      bf16_t hb[4], lb[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float y = oacc[t][r] * inv;
        hb[r] = f2bf_a(y);
        lb[r] = f2bf_a(y - bf2f_a(hb[r]));
      }
      *(uint2*)(orow + t * 16 + 4 * g) =
          make_uint2((uint32_t)hb[0] | ((uint32_t)hb[1] << 16), (uint32_t)hb[2] | ((uint32_t)hb[3] << 16));
      *(uint2*)(orow + o_plane + t * 16 + 4 * g) =
          make_uint2((uint32_t)lb[0] | ((uint32_t)lb[1] << 16), (uint32_t)lb[2] | ((uint32_t)lb[3] << 16));
    }
  } else {
    // unnormalised partial of this key split, merged by k_attn_merge
    const size_t base = ((size_t)split * rows_cap + qrow) * H + h;
    float* orow = ws_o + base * HD;
#pragma unroll
    for (int t = 0; t < HD / 16; ++t)
      *(float4*)(orow + t * 16 + 4 * g) = make_float4(oacc[t][0], oacc[t][1], oacc[t][2], oacc[t][3]);
    if (g == 0) {
      ws_ml[2 * base] = m_run;
      ws_ml[2 * base + 1] = l;
    }
  }
}

// Merge of the key splits (fixed split order): O = sum_s 2^(m_s - M) O_s /
// sum_s 2^(m_s - M) l_s with M = max_s m_s (scores kept in log2 units).
// A workgroup of 256 threads takes 256 / (hd / 4) (row, head) items, each
// thread 4 consecutive dims of one item.
__global__ __launch_bounds__(256) void k_attn_merge(const float* __restrict__ ws_o,
                                                    const float* __restrict__ ws_ml, int kv_splits,
                                                    const int32_t* __restrict__ Mp, int H, int hd,
                                                    int rows_cap, bf16_t* __restrict__ O,
                                                    size_t o_plane) {
  const int tpi = hd / 4;                                   // threads per item
  const int item = blockIdx.x * (256 / tpi) + threadIdx.x / tpi;
  const int e0 = (threadIdx.x % tpi) * 4;
  const int r = item / H, h = item % H;
  if (r >= *Mp) return;
  float M = -INFINITY;
  for (int z = 0; z < kv_splits; ++z) M = fmaxf(M, ws_ml[2 * (((size_t)z * rows_cap + r) * H + h)]);
  float L = 0.f, acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int z = 0; z < kv_splits; ++z) {
    const size_t b = ((size_t)z * rows_cap + r) * H + h;
    const float m = ws_ml[2 * b];
    if (m == -INFINITY) continue;
    const float w = exp2f(m - M);
    L += w * ws_ml[2 * b + 1];
    const float4 o = *(const float4*)(ws_o + b * hd + e0);
    acc[0] += w * o.x; acc[1] += w * o.y; acc[2] += w * o.z; acc[3] += w * o.w;
  }
  bf16_t hb[4], lb[4];
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    const float y = acc[x] / L;
    hb[x] = f2bf_a(y);
    lb[x] = f2bf_a(y - bf2f_a(hb[x]));
  }
  bf16_t* orow = O + ((size_t)r * H + h) * hd + e0;
  *(uint2*)orow = make_uint2((uint32_t)hb[0] | ((uint32_t)hb[1] << 16), (uint32_t)hb[2] | ((uint32_t)hb[3] << 16));
  *(uint2*)(orow + o_plane) =
      make_uint2((uint32_t)lb[0] | ((uint32_t)lb[1] << 16), (uint32_t)lb[2] | ((uint32_t)lb[3] << 16));
}

// fp32 reference-precision kernel for small fp32 models: one wave64 per
// (query row, head); each lane owns head_dim/64 output dims and keys are
// scanned with an online softmax.
__global__ __launch_bounds__(256) void k_attn_f32(const float* __restrict__ Q,
                                                  const float* __restrict__ Kc,
                                                  const float* __restrict__ Vc,
                                                  float* __restrict__ O,
                                                  const int32_t* __restrict__ row_seq,
                                                  const int32_t* __restrict__ row_pos,
                                                  const int32_t* __restrict__ Mp, int H, int Hkv,
                                                  int hd, int maxpos, int B, float scale) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int item = blockIdx.x * 4 + wave;
  const int r = item / H, h = item % H;
  if (r >= *Mp) return;
  const int s = row_seq[r], pos = row_pos[r];
  const int kend = (pos / B + 1) * B;
  const int kv = h / (H / Hkv);
  const float* Kp = Kc + ((size_t)s * Hkv + kv) * (size_t)maxpos * hd;
  const float* Vp = Vc + ((size_t)s * Hkv + kv) * (size_t)maxpos * hd;
  const float* q = Q + ((size_t)r * H + h) * hd;
  const int per = hd / 64;   // 1 or 2
  float qv[2] = {0.f, 0.f}, acc[2] = {0.f, 0.f};
  for (int e = 0; e < per; ++e) qv[e] = q[lane * per + e];
  float m = -INFINITY, l = 0.f;
  for (int j = 0; j < kend; ++j) {
    float part = 0.f;
    for (int e = 0; e < per; ++e) part += qv[e] * Kp[(size_t)j * hd + lane * per + e];
    for (int off = 32; off > 0; off >>= 1) part += __shfl_xor(part, off);
    const float sc = part * scale;
    const float mn = fmaxf(m, sc);
    const float a = expf(m - mn), p = expf(sc - mn);
    l = l * a + p;
    for (int e = 0; e < per; ++e) acc[e] = acc[e] * a + p * Vp[(size_t)j * hd + lane * per + e];
    m = mn;
  }
  float* o = O + (size_t)r * H * hd + h * hd;
  for (int e = 0; e < per; ++e) o[lane * per + e] = acc[e] / l;
}

// waves per workgroup for a window of win_cap rows over a key capacity of
// maxpos (see k_attn_bf16): 8 waves (128 queries per staged K/V tile) where a
// kv head has at least 512 window queries over at least 4096 keys -- the
// long-prefix decode's attention ran 7% faster than with 4 waves (484 -> 449
// ms per decode), the multi-block one (2048 keys) 2.5% slower
static int attention_waves(int win_cap, int H, int Hkv, int maxpos) {
  const int q = (H / Hkv) * win_cap;
  return q <= 32 ? 2 : (q >= 512 && maxpos >= 4096 ? 8 : 4);
}

int attention_splits(int b, int win_cap, int rows_est, int H, int Hkv, int hd, int maxpos) {
  // the launch shape follows win_cap (the largest window); the work estimate
  // follows rows_est, the rows a window usually holds
  const int nw = attention_waves(win_cap, H, Hkv, maxpos);
  const int wgs = (((H / Hkv) * rows_est + 16 * nw - 1) / (16 * nw)) * Hkv * b;
  // workgroups resident per CU (LDS-bound: 37 KB per workgroup at hd 64,
  // 72 KB at hd 128; registers hold the 4-wave hd-64 kind to 3 and the
  // 8-wave kinds to 1): split the key range until
  // the grid fills one resident round of 256 CUs, while every split keeps
  // >= 2 key tiles of the longest range
  const int round = (nw == 8 ? 1 : (hd == 64 ? (nw == 2 ? 4 : 3) : 2)) * 256;
  int splits = 1;
  while (wgs * (splits + 1) <= round && maxpos / (AK * (splits + 1)) >= 2 && splits < 16) ++splits;
  return splits;
}

hipError_t launch_attention(bool is_bf16, const void* Q, size_t q_plane, const KvView& kv,
                            void* O, size_t o_plane, PlanView plan, int b, int win_cap, int H,
                            int Hkv, int hd, int B, int kv_splits, float* ws_o, float* ws_ml,
                            int rows_cap, hipStream_t st) {
  if (is_bf16) {
    if (hd != 64 && hd != 128) return hipErrorInvalidValue;
    if (kv.vstride % 64 || kv.vstride < kv.maxpos) return hipErrorInvalidValue;
    const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)hd));
    const bf16_t* q = (const bf16_t*)Q;
    const bf16_t* k = (const bf16_t*)kv.K;
    const bf16_t* v = (const bf16_t*)kv.V;
    if (kv_splits < 1 || (kv_splits > 1 && (!ws_o || !ws_ml))) return hipErrorInvalidValue;
    const int nw = attention_waves(win_cap, H, Hkv, kv.maxpos);
    const int nqt = ((H / Hkv) * win_cap + 16 * nw - 1) / (16 * nw);
    const int grid = b * Hkv * kv_splits * nqt + 7;
#define BD_ATTN(HD_, NW_)                                                                     \
  k_attn_bf16<HD_, NW_><<<grid, 64 * NW_, 0, st>>>(                                           \
      q, q_plane, k, kv.k_plane, v, kv.v_plane, kv.vstride, (bf16_t*)O, o_plane,              \
      plan.seq_row_start, plan.seq_win_len, plan.seq_win_start, H, Hkv, kv.maxpos, B,         \
      scale_log2, kv_splits, ws_o, ws_ml, rows_cap, b, nqt)
    if (hd == 128) {
      if (nw == 2) BD_ATTN(128, 2); else if (nw == 8) BD_ATTN(128, 8); else BD_ATTN(128, 4);
    } else {
      if (nw == 2) BD_ATTN(64, 2); else if (nw == 8) BD_ATTN(64, 8); else BD_ATTN(64, 4);
    }
#undef BD_ATTN
    if (kv_splits > 1) {
      const int items_per_block = 256 / (hd / 4);
      k_attn_merge<<<(rows_cap * H + items_per_block - 1) / items_per_block, 256, 0, st>>>(
          ws_o, ws_ml, kv_splits, plan.hdr, H, hd, rows_cap, (bf16_t*)O, o_plane);
    }
  } else {
    if (hd != 64 && hd != 128) return hipErrorInvalidValue;
    const int items = rows_cap * H;
    k_attn_f32<<<(items + 3) / 4, 256, 0, st>>>((const float*)Q, (const float*)kv.K, (const float*)kv.V,
                                                (float*)O, plan.row_seq, plan.row_pos, plan.hdr, H,
                                                Hkv, hd, kv.maxpos, B, (float)(1.0 / sqrt((double)hd)));
  }
  return hipGetLastError();
}

}  // namespace bd
