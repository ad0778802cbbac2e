// Row-wise kernels of the denoising step (embedding gather, RMSNorm, RoPE with
// the K/V cache write) and the decode-state kernels (commit/compaction and
// state initialisation).
#include "bd_internal.h"

#include <math.h>

namespace bd {

__device__ __forceinline__ float bf2f_m(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }
__device__ __forceinline__ bf16_t f2bf_m(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

// ------------------------------------------------------------------ embedding
template <bool BF16>
__global__ __launch_bounds__(256) void k_embed(const int32_t* __restrict__ tokens, int tok_stride,
                                               const void* __restrict__ E, int d, int vocab,
                                               const int32_t* __restrict__ hdr,
                                               const int32_t* __restrict__ row_seq,
                                               const int32_t* __restrict__ row_pos,
                                               float* __restrict__ X, int32_t* __restrict__ err) {
  const int r = blockIdx.x;
  if (r >= hdr[0]) return;
  int t = tokens[(size_t)row_seq[r] * tok_stride + row_pos[r]];
  if (t < 0 || t >= vocab) {
    if (threadIdx.x == 0) atomicOr(err, 1);
    t = 0;
  }
  for (int c = threadIdx.x; c < d; c += blockDim.x) {
    float v;
    if constexpr (BF16) v = bf2f_m(((const bf16_t*)E)[(size_t)t * d + c]);
    else v = ((const float*)E)[(size_t)t * d + c];
    X[(size_t)r * d + c] = v;
  }
}

hipError_t launch_embed(bool is_bf16, const int32_t* tokens, int tok_stride, const void* E, int d,
                        int vocab, PlanView plan, int rows_cap, float* X, int32_t* err_flag,
                        hipStream_t st) {
  if (is_bf16)
    k_embed<true><<<rows_cap, 256, 0, st>>>(tokens, tok_stride, E, d, vocab, plan.hdr, plan.row_seq,
                                            plan.row_pos, X, err_flag);
  else
    k_embed<false><<<rows_cap, 256, 0, st>>>(tokens, tok_stride, E, d, vocab, plan.hdr, plan.row_seq,
                                             plan.row_pos, X, err_flag);
  return hipGetLastError();
}

// ------------------------------------------------------------------ RMSNorm
// y = x / sqrt(mean(x^2) + eps) * g in fp32.  Output as fp32 (fp32 models)
// or as the bf16 pair hi = bf16(y), lo = bf16(y - hi) in two planes (bf16
// models: the matmul operand format).  Rows with d % 256 == 0 and d < 2048
// are spread over min(256, d / 4) threads, one to four float4 per thread,
// all loads (x and the pending split partials) in flight at once; the sum of
// squares is reduced in a fixed order (lane shuffles, then the row's waves).
// Rows of 2048 to 4096 (d % 256 == 0) take one wave each, 8 to 16 float4 per
// lane; other widths one wave per row, element by element.
__device__ __forceinline__ void put4(void* out, size_t plane, size_t idx, float4 y, bool pair) {
  if (!pair) {
    *(float4*)((float*)out + idx) = y;
    return;
  }
  const float v[4] = {y.x, y.y, y.z, y.w};
  bf16_t h[4], l[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    h[e] = f2bf_m(v[e]);
    l[e] = f2bf_m(v[e] - bf2f_m(h[e]));
  }
  bf16_t* o = (bf16_t*)out + idx;
  *(uint2*)o = make_uint2((uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16));
  *(uint2*)(o + plane) =
      make_uint2((uint32_t)l[0] | ((uint32_t)l[1] << 16), (uint32_t)l[2] | ((uint32_t)l[3] << 16));
}

template <bool PAIR>
__global__ __launch_bounds__(256) void k_rmsnorm(float* __restrict__ X,
                                                 const float* __restrict__ g, int d, float eps,
                                                 const int32_t* __restrict__ Mp,
                                                 const int32_t* __restrict__ gather,
                                                 void* __restrict__ out, size_t plane,
                                                 ResidSplit fold) {
  __shared__ float red[4];
  const int M = *Mp;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // pending residual split partials: x += p_0 + ... + p_{S-1}, written back
  int S = 1;
  size_t zstride = 0;
  if (fold.ws) {
    const int Mg = *fold.Mp;
    S = resid_splits(Mg, fold);
    zstride = (size_t)((Mg + fold.bm - 1) / fold.bm) * fold.bm * d;
  }
  if (d % 256 == 0 && d >= 2048 && d <= 4096) {
    // wide rows: one wave per row, d / 256 float4 per lane (a row's loads all
    // in flight at once), shuffle-only reduction; split partials added in
    // split order, each split's loads in flight together (multi-block decode:
    // 118 -> 91 ms of RMSNorm per decode against a workgroup per row)
    const int row = blockIdx.x * 4 + wave;
    if (row >= M) return;
    const int src = gather ? gather[row] : row;
    float4* x4 = (float4*)(X + (size_t)src * d);
    const int nv = d >> 8;                     // 8 .. 16
    float4 v[16];
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (i < nv) v[i] = x4[lane + 64 * i];
    if (S > 1) {
      const float4* pz = (const float4*)(fold.ws + (size_t)src * d);
      for (int z = 0; z < S; ++z) {
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (i < nv) {
            const float4 p = pz[z * (zstride >> 2) + lane + 64 * i];
            v[i].x += p.x; v[i].y += p.y; v[i].z += p.z; v[i].w += p.w;
          }
      }
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (i < nv) x4[lane + 64 * i] = v[i];
    }
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (i < nv) ss += v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
    const float inv = 1.0f / sqrtf(ss / (float)d + eps);
    const float4* g4 = (const float4*)g;
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (i < nv) {
        const int c4 = lane + 64 * i;
        const float4 gg = g4[c4];
        const float4 y = make_float4(v[i].x * inv * gg.x, v[i].y * inv * gg.y, v[i].z * inv * gg.z,
                                     v[i].w * inv * gg.w);
        put4(out, plane, (size_t)row * d + 4 * c4, y, PAIR);
      }
    return;
  }
  if (d % 256 == 0 && d <= 4096) {
    const int tpr = min(256, d >> 2);          // threads per row: 64, 128 or 256
    const int rpb = 256 / tpr;
    const int row = blockIdx.x * rpb + (int)threadIdx.x / tpr;
    const int t = (int)threadIdx.x % tpr;
    const int nv = (d >> 2) / tpr;             // float4 per thread, <= 4
    const bool valid = row < M;
    const int src = valid ? (gather ? gather[row] : row) : 0;
    float4* x4 = (float4*)(X + (size_t)src * d);
    float4 v[4];
    float ss = 0.f;
    if (valid) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (i < nv) v[i] = x4[t + i * tpr];
      if (S > 1) {
        const float4* pz = (const float4*)(fold.ws + (size_t)src * d);
        float4 p[4][8];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int z = 0; z < 8; ++z)
            if (i < nv && z < S) p[i][z] = pz[z * (zstride >> 2) + t + i * tpr];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int z = 0; z < 8; ++z)
            if (i < nv && z < S) {
              v[i].x += p[i][z].x; v[i].y += p[i][z].y; v[i].z += p[i][z].z; v[i].w += p[i][z].w;
            }
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (i < nv) x4[t + i * tpr] = v[i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (i < nv) ss += v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
    const int wpr = tpr >> 6;                  // waves per row
    if (wpr > 1) {
      if (lane == 0) red[wave] = ss;
      __syncthreads();
      const int w0 = (wave / wpr) * wpr;
      ss = 0.f;
      for (int w = 0; w < wpr; ++w) ss += red[w0 + w];
    }
    if (!valid) return;
    const float inv = 1.0f / sqrtf(ss / (float)d + eps);
    const float4* g4 = (const float4*)g;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (i < nv) {
        const int c4 = t + i * tpr;
        const float4 gg = g4[c4];
        const float4 y = make_float4(v[i].x * inv * gg.x, v[i].y * inv * gg.y, v[i].z * inv * gg.z,
                                     v[i].w * inv * gg.w);
        put4(out, plane, (size_t)row * d + 4 * c4, y, PAIR);
      }
    return;
  }
  const int row = blockIdx.x * 4 + wave;
  if (row >= M) return;
  const int src = gather ? gather[row] : row;
  float* x = X + (size_t)src * d;
  const float* pz = fold.ws ? fold.ws + (size_t)src * d : nullptr;
  if (S > 1)
    for (int c = lane; c < d; c += 64) {
      float v = x[c];
      for (int z = 0; z < S; ++z) v += pz[z * zstride + c];
      x[c] = v;
    }
  float ss = 0.f;
  for (int c = lane; c < d; c += 64) ss += x[c] * x[c];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  for (int c = lane; c < d; c += 64) {
    const float y = x[c] * inv * g[c];
    if (PAIR) {
      const bf16_t h = f2bf_m(y);
      ((bf16_t*)out)[(size_t)row * d + c] = h;
      ((bf16_t*)out)[(size_t)row * d + c + plane] = f2bf_m(y - bf2f_m(h));
    } else {
      ((float*)out)[(size_t)row * d + c] = y;
    }
  }
}

hipError_t launch_rmsnorm(bool is_bf16, float* X, const float* g, int d, float eps,
                          const int32_t* M_dev, const int32_t* gather, int rows_cap, void* out,
                          size_t out_plane, const ResidSplit& fold, hipStream_t st) {
  // rows per block: 4 (a wave per row) for wide rows and widths off the
  // float4 paths, else 256 threads over 256 / (d / 4) rows
  const int rpb = (d % 256 == 0 && d < 2048) ? 256 / min(256, d >> 2) : 4;
  const int blocks = (rows_cap + rpb - 1) / rpb;
  if (is_bf16)
    k_rmsnorm<true><<<blocks, 256, 0, st>>>(X, g, d, eps, M_dev, gather, out, out_plane, fold);
  else
    k_rmsnorm<false><<<blocks, 256, 0, st>>>(X, g, d, eps, M_dev, gather, out, 0, fold);
  return hipGetLastError();
}

// ------------------------------------------------------------------ RoPE + KV
// fp32 models: rotate-half RoPE of q and k at the row's absolute position
// (angle and rotation in fp64, one rounding to fp32); q -> Q[row][head][hd],
// k and v -> the layer's cache slots [seq][kv head][pos][hd].  (bf16 models
// do this in the QKV GEMM epilogue.)
__global__ __launch_bounds__(256) void k_rope_kv(const float* __restrict__ QKV,
                                                 const int32_t* __restrict__ hdr,
                                                 const int32_t* __restrict__ row_seq,
                                                 const int32_t* __restrict__ row_pos, int H, int Hkv,
                                                 int hd, const double* __restrict__ inv_freq,
                                                 float* __restrict__ Q, KvView kv) {
  const int r = blockIdx.x;
  if (r >= hdr[0]) return;
  const int s = row_seq[r], pos = row_pos[r];
  const int half = hd / 2, qkv = (H + 2 * Hkv) * hd;
  const float* src = QKV + (size_t)r * qkv;
  float* K = (float*)kv.K;
  float* V = (float*)kv.V;
  for (int idx = threadIdx.x; idx < (H + Hkv) * half; idx += blockDim.x) {
    const int head = idx / half, i = idx % half;
    double sn, cs;
    sincos((double)pos * inv_freq[i], &sn, &cs);
    const double x1 = src[head * hd + i], x2 = src[head * hd + i + half];
    const float y1 = (float)(x1 * cs - x2 * sn), y2 = (float)(x2 * cs + x1 * sn);
    float* o = (head < H) ? Q + ((size_t)r * H + head) * hd
                          : K + (((size_t)s * Hkv + (head - H)) * kv.maxpos + pos) * hd;
    o[i] = y1;
    o[i + half] = y2;
  }
  for (int idx = threadIdx.x; idx < Hkv * hd; idx += blockDim.x) {
    const int kh = idx / hd, e = idx % hd;
    V[(((size_t)s * Hkv + kh) * kv.maxpos + pos) * hd + e] = src[(H + Hkv) * hd + idx];
  }
}

hipError_t launch_rope_kv(const float* QKV, PlanView plan, int rows_cap, int H, int Hkv, int hd,
                          const double* inv_freq, float* Q, const KvView& kv, hipStream_t st) {
  k_rope_kv<<<rows_cap, 256, 0, st>>>(QKV, plan.hdr, plan.row_seq, plan.row_pos, H, Hkv, hd, inv_freq,
                                      Q, kv);
  return hipGetLastError();
}

// ------------------------------------------------------------------ commit
constexpr int MAXB = 256;     // sequences per state
constexpr int MAXNB = 8;      // in-flight blocks per sequence

__device__ __forceinline__ int wave_popc(bool p) { return __popcll(__ballot(p)); }

// Single workgroup; wave w owns sequences w, w + 16, ...
//  phase 1: commit rule, token/commit-step writes, per-block resolution counts,
//           cache write of the pending blocks, in-order sweep, admission,
//           the blocks the next forward takes, participation counts;
//  phase 2: prefix sums of the next window sizes and masked-row counts;
//  phase 3: the next step plan (rows = [pending blocks][forwarded active
//           blocks], masked rows ascending).
// The forwarded active blocks are always the first n_fwd of the active list:
// all of them, or under the static skip rule the oldest one and the ones
// after it that already hold a resolved position (a fully masked block can
// only gain one by being forwarded, so they form a prefix).
__global__ __launch_bounds__(1024) void k_commit(CommitArgs a) {
  __shared__ int s_win[MAXB], s_lm[MAXB], s_rs[MAXB], s_ls[MAXB];
  __shared__ int s_cl[MAXB], s_fa[MAXB], s_sw[MAXB], s_nf[MAXB], s_full0[MAXB], s_nfull[MAXB], s_lmn[MAXB],
      s_lm0[MAXB];
  __shared__ long long s_pairs[MAXB], s_keys[MAXB];
  __shared__ int s_ncommit[MAXB];
  __shared__ int s_part[MAXB][6];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, nw = blockDim.x >> 6;
  const int P = a.P, G = a.G, B = a.B;

  for (int s = wave; s < a.b; s += nw) {
    int* ss = a.seq_state + s * SS_N;
    const int done = ss[SS_DONE];
    const int lm0 = a.in.seq_lm_start[s];
    const int lmn = done ? 0 : a.in.seq_lm_cnt[s];
    int cache_len = ss[SS_CACHE_LEN], n_pend = ss[SS_N_PEND], first_act = ss[SS_FIRST_ACT];
    int n_act = ss[SS_N_ACT], next_blk = ss[SS_NEXT_BLK];
    const int n_fwd = ss[SS_N_FWD];
    if (done) {
      if (lane == 0) {
        s_win[s] = 0; s_lm[s] = 0; s_cl[s] = cache_len; s_fa[s] = first_act; s_sw[s] = 0;
        s_nf[s] = 0; s_full0[s] = 0; s_nfull[s] = 0; s_lmn[s] = 0; s_lm0[s] = lm0;
        s_pairs[s] = 0; s_keys[s] = 0; s_ncommit[s] = 0;
        for (int q = 0; q < 6; ++q) s_part[s][q] = 0;
      }
      continue;
    }
    // work of the forward just executed: visible query-key pairs (per head)
    // and keys streamed (prefix + window, per kv head)
    if (lane == 0) {
      const long long start = a.in.seq_win_start[s], nbw = a.in.seq_win_len[s] / B;
      s_pairs[s] = (long long)B * (nbw * start + (long long)B * nbw * (nbw + 1) / 2);
      s_keys[s] = start + (long long)a.in.seq_win_len[s];
    }
    // pass 1, per active block k: masked positions, whether one clears tau,
    // and the most confident one (lowest position among equals)
    int blk_masked[MAXNB], blk_commit[MAXNB], blk_best_pos[MAXNB];
    float blk_best[MAXNB];
    bool blk_any[MAXNB];
#pragma unroll
    for (int k = 0; k < MAXNB; ++k) {
      blk_masked[k] = 0; blk_commit[k] = 0; blk_best[k] = -INFINITY; blk_best_pos[k] = 0x7fffffff;
      blk_any[k] = false;
    }
    for (int base = 0; base < lmn; base += 64) {
      const int i = base + lane;
      const bool valid = i < lmn;
      float cf = -INFINITY;
      int pos = 0x7fffffff, kb = -1;
      if (valid) {
        cf = a.conf[lm0 + i];
        pos = a.in.row_pos[a.in.lm_row[lm0 + i]];
        kb = (pos - P) / B - first_act;
      }
#pragma unroll
      for (int k = 0; k < MAXNB; ++k) {
        if (k >= n_fwd) break;                 // wave-uniform
        const bool mine = valid && kb == k;
        blk_masked[k] += wave_popc(mine);
        blk_any[k] |= mine && cf >= a.tau;
        if (mine && (cf > blk_best[k] || (cf == blk_best[k] && pos < blk_best_pos[k]))) {
          blk_best[k] = cf;
          blk_best_pos[k] = pos;
        }
      }
    }
#pragma unroll
    for (int k = 0; k < MAXNB; ++k) {
      if (k >= n_fwd) break;
      blk_any[k] = __ballot(blk_any[k]) != 0;
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const float ob = __shfl_xor(blk_best[k], off);
        const int op = __shfl_xor(blk_best_pos[k], off);
        if (ob > blk_best[k] || (ob == blk_best[k] && op < blk_best_pos[k])) {
          blk_best[k] = ob;
          blk_best_pos[k] = op;
        }
      }
    }
    // blocks left out of the forward are fully masked
#pragma unroll
    for (int k = 0; k < MAXNB; ++k)
      if (k >= n_fwd && k < n_act) blk_masked[k] = B;
    // forced commits.  Semi-completion off: one per sequence when no position
    // clears tau, the most confident over all blocks (blocks are in position
    // order, so the first block holding the maximum has its lowest position).
    // On: one per fully activated block with masked positions of which none
    // clears tau; block k > 0 is fully activated when block k - 1 had
    // resolved >= semi_min positions at the start of the step.
    int forced_pos[MAXNB];
#pragma unroll
    for (int k = 0; k < MAXNB; ++k) forced_pos[k] = -1;
    if (a.semi_min < 0) {
      bool any = false;
      float best = -INFINITY;
      int bp = -1;
#pragma unroll
      for (int k = 0; k < MAXNB; ++k) {
        any |= blk_any[k];
        if (k < n_fwd && blk_masked[k] > 0 && (bp < 0 || blk_best[k] > best)) {
          best = blk_best[k];
          bp = blk_best_pos[k];
        }
      }
      if (!any) forced_pos[0] = bp;
    } else {
#pragma unroll
      for (int k = 0; k < MAXNB; ++k) {
        const bool full = k == 0 || (B - blk_masked[k > 0 ? k - 1 : 0]) >= a.semi_min;
        if (k < n_fwd && blk_masked[k] > 0 && full && !blk_any[k]) forced_pos[k] = blk_best_pos[k];
      }
    }
    // pass 2: commit, and count committed positions per active block
    for (int base = 0; base < lmn; base += 64) {
      const int i = base + lane;
      const bool valid = i < lmn;
      bool c = false;
      int kb = -1;
      if (valid) {
        const float cf = a.conf[lm0 + i];
        const int pos = a.in.row_pos[a.in.lm_row[lm0 + i]];
        c = cf >= a.tau;
#pragma unroll
        for (int k = 0; k < MAXNB; ++k) c |= pos == forced_pos[k];
        kb = (pos - P) / B - first_act;
        if (c) {
          a.tokens[(size_t)s * a.tok_stride + pos] = a.tok[lm0 + i];
          a.commit_step[(size_t)s * G + pos - P] = a.step;
        }
        a.commit_flag[lm0 + i] = c ? 1 : 0;
      }
#pragma unroll
      for (int k = 0; k < MAXNB; ++k) {
        if (k >= n_act) break;
        blk_commit[k] += wave_popc(valid && kb == k && c);
      }
    }
    int ncommit = 0;
#pragma unroll
    for (int k = 0; k < MAXNB; ++k) ncommit += blk_commit[k];
    // the blocks that rode along as clean rows now hold their K/V
    cache_len += n_pend * B;
    // in-order sweep: commit a chain of complete blocks from the oldest
    int sw = 0;
#pragma unroll
    for (int k = 0; k < MAXNB; ++k)
      if (sw == k && k < n_act && blk_masked[k] == blk_commit[k]) sw = k + 1;
    const int first_act_old = first_act, n_act_old = n_act;
    first_act += sw;
    n_act -= sw;
    const int nblk = G / B;
    // admission: the youngest active block after the sweep is pre-sweep
    // block sw + n_act - 1; a newly admitted block has nothing resolved
    int young = 0;
#pragma unroll
    for (int k = 0; k < MAXNB; ++k)
      if (k == sw + n_act - 1) young = B - (blk_masked[k] - blk_commit[k]);
    while (n_act < a.nb && next_blk < nblk && (n_act == 0 || young >= a.add_min)) {
      ++n_act; ++next_blk;
      young = 0;
    }
    const int now_done = (n_act == 0);
    // blocks of the next forward: pre-sweep blocks sw .. sw + nf - 1, those
    // past n_act_old being newly admitted (fully masked)
    int nf = n_act;
    if (a.skip && n_act > 0) {
      nf = 1;
      bool run = true;
#pragma unroll
      for (int k = 0; k < MAXNB; ++k) {
        if (run && k > sw && k < n_act_old) {
          if (blk_masked[k] - blk_commit[k] < B) ++nf;
          else run = false;
        }
      }
    }
    // masked rows of the next forward: the unresolved positions of blocks
    // forwarded this step, then whole blocks that were not
    int left = 0;
#pragma unroll
    for (int k = 0; k < MAXNB; ++k)
      if (k >= sw && k < sw + nf && k < n_fwd) left += blk_masked[k] - blk_commit[k];
    const int full0 = sw > n_fwd ? sw : n_fwd;
    const int nfull = sw + nf - full0 > 0 ? sw + nf - full0 : 0;
    // participation of the forward just executed
    int p_zero = 0, p_save = 0, p_defer = 0;
#pragma unroll
    for (int k = 0; k < MAXNB; ++k) {
      if (k < n_fwd) {
        p_zero += blk_commit[k] == 0;
        if (k > 0 && blk_masked[k] == B) {
          if (blk_commit[k] == 0) ++p_save;
          else ++p_defer;
        }
      }
    }
    if (lane == 0) {
      ss[SS_CACHE_LEN] = cache_len;
      ss[SS_N_PEND] = sw;
      ss[SS_FIRST_ACT] = first_act;
      ss[SS_N_ACT] = n_act;
      ss[SS_NEXT_BLK] = next_blk;
      ss[SS_DONE] = now_done;
      ss[SS_FORWARDS] += 1;
      ss[SS_N_FWD] = now_done ? 0 : nf;
      s_win[s] = now_done ? 0 : (sw + nf) * B;
      s_lm[s] = now_done ? 0 : left + nfull * B;
      s_cl[s] = cache_len; s_fa[s] = first_act_old; s_sw[s] = sw; s_nf[s] = nf;
      s_full0[s] = first_act_old + full0; s_nfull[s] = now_done ? 0 : nfull;
      s_lmn[s] = now_done ? 0 : lmn; s_lm0[s] = lm0;
      s_ncommit[s] = ncommit;
      s_part[s][0] = n_fwd; s_part[s][1] = p_zero; s_part[s][2] = p_save; s_part[s][3] = p_defer;
      s_part[s][4] = n_pend; s_part[s][5] = n_act_old - n_fwd;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int r = 0, l = 0;
    for (int s = 0; s < a.b; ++s) {
      s_rs[s] = r; s_ls[s] = l;
      r += s_win[s]; l += s_lm[s];
    }
    a.out.hdr[0] = r;
    a.out.hdr[1] = l;
    a.out.hdr[2] = (r == 0) ? 1 : 0;
    long long pairs = 0, keys = 0, nc = 0;
    for (int s = 0; s < a.b; ++s) { pairs += s_pairs[s]; keys += s_keys[s]; nc += s_ncommit[s]; }
    const int m_in = a.in.hdr[0];
    a.stats[0] += (m_in > 0);
    a.stats[1] += m_in;
    a.stats[2] += a.in.hdr[1];
    a.stats[3] += pairs;
    a.stats[4] += keys;
    a.stats[5] += nc;
    for (int q = 0; q < 6; ++q) {
      long long t = 0;
      for (int s = 0; s < a.b; ++s) t += s_part[s][q];
      a.stats[6 + q] += t;
    }
  }
  __syncthreads();
  for (int s = wave; s < a.b; s += nw) {
    const int rs = s_rs[s], W = s_win[s], cl = s_cl[s], ls = s_ls[s];
    if (lane == 0) {
      a.out.seq_row_start[s] = rs; a.out.seq_win_len[s] = W; a.out.seq_win_start[s] = cl;
      a.out.seq_lm_start[s] = ls; a.out.seq_lm_cnt[s] = s_lm[s];
    }
    for (int e = lane; e < W; e += 64) {
      a.out.row_seq[rs + e] = s;
      a.out.row_pos[rs + e] = cl + e;
    }
    const int lmn = s_lmn[s], lm0 = s_lm0[s], fa = s_fa[s], sw = s_sw[s], nf = s_nf[s];
    int w = 0;
    for (int base = 0; base < lmn; base += 64) {
      const int i = base + lane;
      bool keep = false;
      int pos = 0;
      if (i < lmn) {
        pos = a.in.row_pos[a.in.lm_row[lm0 + i]];
        const int kb = (pos - P) / B - fa;
        keep = !a.commit_flag[lm0 + i] && kb >= sw && kb < sw + nf;
      }
      const unsigned long long m = __ballot(keep);
      const int pre = __popcll(m & ((1ull << lane) - 1ull));
      if (keep) a.out.lm_row[ls + w + pre] = rs + (pos - cl);
      w += __popcll(m);
    }
    const int nfull = s_nfull[s], p0 = P + s_full0[s] * B;
    for (int e = lane; e < nfull * B; e += 64) a.out.lm_row[ls + w + e] = rs + (p0 + e - cl);
  }
}

hipError_t launch_commit(const CommitArgs& a, hipStream_t st) {
  if (a.b > MAXB || a.nb > MAXNB) return hipErrorInvalidValue;
  k_commit<<<1, 1024, 0, st>>>(a);
  return hipGetLastError();
}

// ------------------------------------------------------------------ init
__global__ __launch_bounds__(1024) void k_init_decode(InitArgs a) {
  __shared__ int s_win[MAXB], s_rs[MAXB];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, nw = blockDim.x >> 6;
  const int stride = a.P + a.G, nblk = a.G / a.B;
  // admission as after a commit: the first block unconditionally, further
  // ones while the youngest (nothing resolved yet) reaches add_min
  int nact = min(1, nblk);
  while (nact < a.nb && nact < nblk && 0 >= a.add_min) ++nact;
  const int nfwd = a.skip ? min(nact, 1) : nact;     // admitted blocks are fully masked
  for (int s = wave; s < a.b; s += nw) {
    int32_t* t = a.tokens + (size_t)s * stride;
    if (a.prompt) {
      for (int j = lane; j < a.P; j += 64) {
        const int v = a.prompt[(size_t)s * a.P + j];
        if (v < 0 || v >= a.vocab) atomicOr(a.err_flag, 1);
        t[j] = v;
      }
    }
    for (int j = lane; j < a.G; j += 64) {
      t[a.P + j] = a.mask_id;
      a.commit_step[(size_t)s * a.G + j] = -1;
    }
    if (lane == 0) {
      int32_t* ss = a.seq_state + s * SS_N;
      ss[SS_CACHE_LEN] = a.P; ss[SS_N_PEND] = 0; ss[SS_FIRST_ACT] = 0; ss[SS_N_ACT] = nact;
      ss[SS_NEXT_BLK] = nact; ss[SS_DONE] = 0; ss[SS_FORWARDS] = 0; ss[SS_N_FWD] = nfwd;
      s_win[s] = nfwd * a.B;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int r = 0;
    for (int s = 0; s < a.b; ++s) { s_rs[s] = r; r += s_win[s]; }
    a.plan.hdr[0] = r; a.plan.hdr[1] = r; a.plan.hdr[2] = (r == 0);
    for (int k = 0; k < BD_NSTATS; ++k) a.stats[k] = 0;
    if (a.prefill.hdr) {
      a.prefill.hdr[0] = a.b * a.P; a.prefill.hdr[1] = 0; a.prefill.hdr[2] = 0;
    }
  }
  __syncthreads();
  for (int s = wave; s < a.b; s += nw) {
    const int rs = s_rs[s], W = s_win[s];
    if (lane == 0) {
      a.plan.seq_row_start[s] = rs; a.plan.seq_win_len[s] = W; a.plan.seq_win_start[s] = a.P;
      a.plan.seq_lm_start[s] = rs; a.plan.seq_lm_cnt[s] = W;
      if (a.prefill.hdr) {
        a.prefill.seq_row_start[s] = s * a.P; a.prefill.seq_win_len[s] = a.P;
        a.prefill.seq_win_start[s] = 0; a.prefill.seq_lm_start[s] = 0; a.prefill.seq_lm_cnt[s] = 0;
      }
    }
    for (int e = lane; e < W; e += 64) {
      a.plan.row_seq[rs + e] = s;
      a.plan.row_pos[rs + e] = a.P + e;
      a.plan.lm_row[rs + e] = rs + e;
    }
    if (a.prefill.hdr) {
      for (int j = lane; j < a.P; j += 64) {
        a.prefill.row_seq[s * a.P + j] = s;
        a.prefill.row_pos[s * a.P + j] = j;
      }
    }
  }
}

hipError_t launch_init_decode(const InitArgs& a, hipStream_t st) {
  if (a.b > MAXB) return hipErrorInvalidValue;
  k_init_decode<<<1, 1024, 0, st>>>(a);
  return hipGetLastError();
}

// ------------------------------------------------------------------ fp8 weights
// Nearest E4M3 code (ties to even) of |v| <= 448: the spacing of representable
// values is 2^(floor(log2|v|) - 3) from the smallest normal 2^-6 up and 2^-9
// below it; the rounded magnitude is then split into exponent and mantissa
// fields (rounding may have carried it into the next binade).  All steps
// are exact in fp32 except the one rounding of rintf.
__device__ __forceinline__ uint32_t e4m3_code(float v) {
  const float a = fabsf(v);
  uint32_t code = 0;
  if (a > 0.f) {
    int ea;
    (void)frexpf(a, &ea);                       // a = f 2^ea, 0.5 <= f < 1
    const int qe = a >= 0x1p-6f ? ea - 4 : -9;
    const float q = ldexpf(rintf(ldexpf(a, -qe)), qe);
    if (q >= 0x1p-6f) {
      int eq;
      (void)frexpf(q, &eq);
      code = ((uint32_t)(eq + 6) << 3) | (uint32_t)(ldexpf(q, 1 - eq) * 8.0f - 8.0f);
    } else {
      code = (uint32_t)ldexpf(q, 9);
    }
  }
  return v < 0.f ? (code | 0x80u) : code;
}

// One workgroup per row: the row's largest magnitude gives the scale 2^E
// with E the smallest integer such that amax / 2^E <= 448 (amax = f 2^x,
// 448 = 0.875 2^9: E = x - 9, or x - 8 when f > 0.875; 0 for a zero row),
// then every element is coded as w / 2^E.
__global__ __launch_bounds__(256) void k_quant_fp8_rows(const bf16_t* __restrict__ W, int cols,
                                                        uint8_t* __restrict__ Q, float* __restrict__ scale) {
  __shared__ float red[4];
  const size_t row = blockIdx.x;
  const bf16_t* w = W + row * cols;
  float amax = 0.f;
  for (int c = threadIdx.x; c < cols; c += 256) amax = fmaxf(amax, fabsf(bf2f_m(w[c])));
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = amax;
  __syncthreads();
  amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  int E = 0;
  if (amax > 0.f) {
    int x;
    const float f = frexpf(amax, &x);
    E = x - 9 + (f > 0.875f ? 1 : 0);
  }
  for (int c = threadIdx.x; c < cols; c += 256) Q[row * cols + c] = (uint8_t)e4m3_code(ldexpf(bf2f_m(w[c]), -E));
  if (threadIdx.x == 0) scale[row] = ldexpf(1.0f, E);
}

hipError_t launch_quant_fp8_rows(const void* W, int rows, int cols, uint8_t* Q, float* scale, hipStream_t st) {
  if (rows < 1 || cols < 1) return hipErrorInvalidValue;
  k_quant_fp8_rows<<<rows, 256, 0, st>>>((const bf16_t*)W, cols, Q, scale);
  return hipGetLastError();
}

// ------------------------------------------------------------------ MXFP4 weights
// Nearest E2M1 code (ties to even, magnitudes above 6 saturating): the
// spacing of representable values is 2^(floor(log2|v|) - 1) from 1 up and 0.5
// below; the rounded magnitude q (at most 6) is then split into exponent and
// mantissa fields.  Exact in fp32 except the one rounding of rintf.
__device__ __forceinline__ uint32_t e2m1_code(float v) {
  const float a = fabsf(v);
  uint32_t code = 0;
  if (a > 0.f) {
    int ea;
    (void)frexpf(a, &ea);                       // a = f 2^ea, 0.5 <= f < 1
    const int qe = a >= 1.f ? ea - 2 : -1;
    const float q = fminf(ldexpf(rintf(ldexpf(a, -qe)), qe), 6.f);
    if (q >= 1.f) {
      int eq;
      (void)frexpf(q, &eq);
      code = ((uint32_t)eq << 1) | (uint32_t)(ldexpf(q, 2 - eq) - 2.f);
    } else {
      code = (uint32_t)(q * 2.f);
    }
  }
  return v < 0.f ? (code | 8u) : code;
}

// One thread per (row group, block, row): the block's largest magnitude
// amax = f 2^x gives the exponent X = x - 3 = floor(log2 amax) - 2 (-127 for
// a zero block; clamped to E8M0's [-127, 127]), then each element is coded as
// w / 2^X (exact: a power-of-two scaling of a bf16 value).  Threads of
// consecutive rows write consecutive 16-byte code rows.
__global__ __launch_bounds__(256) void k_quant_mxfp4_rows(const bf16_t* __restrict__ W, int rows, int cols,
                                                          int group_rows, uint8_t* __restrict__ codes,
                                                          uint8_t* __restrict__ exps) {
  const int nb = cols / MX_BLOCK;
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (size_t)rows * nb) return;
  const int r = (int)(idx % group_rows);
  const size_t gk = idx / group_rows;             // g * nb + kb
  const int kb = (int)(gk % nb), g = (int)(gk / nb);
  const bf16_t* w = W + ((size_t)g * group_rows + r) * cols + (size_t)kb * MX_BLOCK;
  float v[MX_BLOCK];
  float amax = 0.f;
#pragma unroll
  for (int j = 0; j < MX_BLOCK; ++j) {
    v[j] = bf2f_m(w[j]);
    amax = fmaxf(amax, fabsf(v[j]));
  }
  int X = -127;
  if (amax > 0.f) {
    int x;
    (void)frexpf(amax, &x);
    X = x - 3;
    X = X < -127 ? -127 : (X > 127 ? 127 : X);
  }
  uint32_t packed[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int j = 0; j < MX_BLOCK; ++j) packed[j >> 3] |= e2m1_code(ldexpf(v[j], -X)) << (4 * (j & 7));
  *(uint4*)(codes + idx * 16) = make_uint4(packed[0], packed[1], packed[2], packed[3]);
  exps[idx] = (uint8_t)(X + 127);
}

hipError_t launch_quant_mxfp4_rows(const void* W, int rows, int cols, int group_rows, uint8_t* codes,
                                   uint8_t* exps, hipStream_t st) {
  if (rows < 1 || cols < MX_BLOCK || cols % MX_BLOCK || group_rows < 1 || rows % group_rows)
    return hipErrorInvalidValue;
  const size_t n = (size_t)rows * (cols / MX_BLOCK);
  k_quant_mxfp4_rows<<<(unsigned)((n + 255) / 256), 256, 0, st>>>((const bf16_t*)W, rows, cols, group_rows, codes,
                                                                  exps);
  return hipGetLastError();
}

// ------------------------------------------------------------------ debug
__global__ void k_scatter_logits(const float* __restrict__ logits, const int32_t* __restrict__ hdr,
                                 const int32_t* __restrict__ lm_row,
                                 const int32_t* __restrict__ row_seq,
                                 const int32_t* __restrict__ row_pos, int V, int P, int G,
                                 float* __restrict__ out) {
  const int i = blockIdx.y;
  if (i >= hdr[1]) return;
  const int r = lm_row[i];
  const size_t o = ((size_t)row_seq[r] * G + (row_pos[r] - P)) * V;
  for (int n = blockIdx.x * blockDim.x + threadIdx.x; n < V; n += gridDim.x * blockDim.x)
    out[o + n] = logits[(size_t)i * V + n];
}

hipError_t launch_scatter_logits(const float* logits, PlanView plan, int V, int P, int G,
                                 float* out, int lm_cap, hipStream_t st) {
  k_scatter_logits<<<dim3((V + 2047) / 2048, lm_cap), 256, 0, st>>>(logits, plan.hdr, plan.lm_row,
                                                                     plan.row_seq, plan.row_pos, V,
                                                                     P, G, out);
  return hipGetLastError();
}

__global__ void k_scatter_stats(const float* __restrict__ conf, const int32_t* __restrict__ tok,
                                const int32_t* __restrict__ hdr, const int32_t* __restrict__ lm_row,
                                const int32_t* __restrict__ row_seq,
                                const int32_t* __restrict__ row_pos, int P, int G,
                                float* __restrict__ dconf, int32_t* __restrict__ dtok) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= hdr[1]) return;
  const int r = lm_row[i];
  const size_t o = (size_t)row_seq[r] * G + (row_pos[r] - P);
  if (dconf) dconf[o] = conf[i];
  if (dtok) dtok[o] = tok[i];
}

hipError_t launch_scatter_stats(const float* conf, const int32_t* tok, PlanView plan, int P, int G,
                                float* dconf, int32_t* dtok, int lm_cap, hipStream_t st) {
  k_scatter_stats<<<(lm_cap + 255) / 256, 256, 0, st>>>(conf, tok, plan.hdr, plan.lm_row, plan.row_seq,
                                                        plan.row_pos, P, G, dconf, dtok);
  return hipGetLastError();
}

// Pack gate and up projections into groups of 16 rows: packed rows
// [32q, 32q + 16) = gate rows [16q, 16q + 16), [32q + 16, 32q + 32) = up rows.
__global__ void k_pack_gate_up(const uint8_t* __restrict__ gate, const uint8_t* __restrict__ up,
                               uint8_t* __restrict__ out, size_t row_bytes) {
  const int pr = blockIdx.x;
  const int q = pr >> 5, w = pr & 31;
  const uint8_t* src = (w < 16 ? gate : up) + (size_t)(q * 16 + (w & 15)) * row_bytes;
  uint8_t* dst = out + (size_t)pr * row_bytes;
  for (size_t c = threadIdx.x * 4; c < row_bytes; c += blockDim.x * 4)
    *(uint32_t*)(dst + c) = *(const uint32_t*)(src + c);
}

hipError_t launch_pack_gate_up(const void* gate, const void* up, void* out, int F, size_t row_bytes,
                               hipStream_t st) {
  if (F % 16 || row_bytes % 4) return hipErrorInvalidValue;
  k_pack_gate_up<<<2 * F, 256, 0, st>>>((const uint8_t*)gate, (const uint8_t*)up, (uint8_t*)out,
                                        row_bytes);
  return hipGetLastError();
}

// Pair-interleave the q and k head rows of a QKV weight: in each head,
// packed row 2i <- dim i, 2i + 1 <- dim i + hd/2.  v rows are copied as is.
__global__ void k_permute_qk_rows(const uint8_t* __restrict__ W, uint8_t* __restrict__ out, int qk_rows,
                                  int hd, size_t row_bytes) {
  const int pr = blockIdx.x;
  int src = pr;
  if (pr < qk_rows) {
    const int head = pr / hd, cp = pr % hd;
    src = head * hd + ((cp & 1) ? (cp >> 1) + hd / 2 : (cp >> 1));
  }
  const uint8_t* s = W + (size_t)src * row_bytes;
  uint8_t* d = out + (size_t)pr * row_bytes;
  for (size_t c = threadIdx.x * 4; c < row_bytes; c += blockDim.x * 4)
    *(uint32_t*)(d + c) = *(const uint32_t*)(s + c);
}

hipError_t launch_permute_qk_rows(const void* W, void* out, int H, int Hkv, int hd, size_t row_bytes,
                                  hipStream_t st) {
  if (hd % 2 || row_bytes % 4) return hipErrorInvalidValue;
  k_permute_qk_rows<<<(H + 2 * Hkv) * hd, 256, 0, st>>>((const uint8_t*)W, (uint8_t*)out,
                                                        (H + Hkv) * hd, hd, row_bytes);
  return hipGetLastError();
}

// cos/sin of pos * inv_freq[i] in fp64 (the angle and its sine and cosine
// computed as in k_rope_kv).
__global__ void k_rope_table(const double* __restrict__ inv_freq, int half, int maxpos,
                             double* __restrict__ tab) {
  const int pos = blockIdx.x;
  for (int i = threadIdx.x; i < half; i += blockDim.x) {
    double sn, cs;
    sincos((double)pos * inv_freq[i], &sn, &cs);
    tab[((size_t)pos * half + i) * 2] = cs;
    tab[((size_t)pos * half + i) * 2 + 1] = sn;
  }
}

hipError_t launch_rope_table(const double* inv_freq, int hd, int maxpos, double* tab, hipStream_t st) {
  if (maxpos < 1) return hipSuccess;
  k_rope_table<<<maxpos, 64, 0, st>>>(inv_freq, hd / 2, maxpos, tab);
  return hipGetLastError();
}


// Zero n 32-bit words (a kernel, so that the clear can sit in a captured
// stream; 16-byte stores on the aligned body).
__global__ __launch_bounds__(256) void k_zero_words(uint32_t* __restrict__ p, size_t n) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  const size_t i0 = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t head = ((16 - ((uintptr_t)p & 15)) & 15) / 4;     // words before a 16-byte boundary
  const size_t h = head < n ? head : n;
  if (i0 < h) p[i0] = 0u;
  u32x4* q = (u32x4*)(p + h);
  const size_t nv = (n - h) / 4;
  for (size_t i = i0; i < nv; i += stride) q[i] = u32x4{0u, 0u, 0u, 0u};
  for (size_t i = h + 4 * nv + i0; i < n; i += stride) p[i] = 0u;
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t st) {
  if (bytes == 0) return hipSuccess;
  if (((uintptr_t)p & 3) || (bytes & 3)) return hipErrorInvalidValue;
  const size_t n = bytes / 4;
  size_t blocks = (n / 4 + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  k_zero_words<<<(unsigned)blocks, 256, 0, st>>>((uint32_t*)p, n);
  return hipGetLastError();
}

}  // namespace bd
