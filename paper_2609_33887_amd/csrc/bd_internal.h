// Internal declarations shared by the HIP sources of the block-diffusion
// library (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bd {

typedef uint16_t bf16_t;   // bfloat16 bit pattern in memory
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
// native 16-byte vector (HIP's uint4 is a struct, which keeps register arrays
// of it on the stack)
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Per-sequence decode descriptor, int32 fields of seq_state[b][SS_N].
enum {
  SS_CACHE_LEN = 0,   // positions [0, cache_len) hold K/V from clean tokens
  SS_N_PEND = 1,      // committed blocks awaiting their cache write
  SS_FIRST_ACT = 2,   // generation-block index of the first active block
  SS_N_ACT = 3,       // active blocks
  SS_NEXT_BLK = 4,    // first block not yet admitted
  SS_DONE = 5,
  SS_FORWARDS = 6,
  SS_N_FWD = 7,       // active blocks the next forward takes (the first ones)
  SS_N = 8
};

// Step plan: which rows the next forward runs and which get an LM head.
// Layout inside one int32 buffer (see plan_* helpers).
struct PlanView {
  int32_t* hdr;          // [0] = M rows, [1] = M_lm rows, [2] = all_done
  int32_t* row_seq;      // [rows_cap]
  int32_t* row_pos;      // [rows_cap] absolute position of the row
  int32_t* lm_row;       // [lm_cap]   index into rows, ascending
  int32_t* seq_row_start;  // [b]
  int32_t* seq_win_len;    // [b]
  int32_t* seq_win_start;  // [b] absolute position of the first window row
  int32_t* seq_lm_start;   // [b]
  int32_t* seq_lm_cnt;     // [b]
};

inline size_t plan_words(int rows_cap, int lm_cap, int b) {
  return 16 + 2 * (size_t)rows_cap + (size_t)lm_cap + 5 * (size_t)b;
}

inline PlanView plan_view(int32_t* base, int rows_cap, int lm_cap, int b) {
  PlanView p;
  p.hdr = base;
  p.row_seq = base + 16;
  p.row_pos = p.row_seq + rows_cap;
  p.lm_row = p.row_pos + rows_cap;
  p.seq_row_start = p.lm_row + lm_cap;
  p.seq_win_len = p.seq_row_start + b;
  p.seq_win_start = p.seq_win_len + b;
  p.seq_lm_start = p.seq_win_start + b;
  p.seq_lm_cnt = p.seq_lm_start + b;
  return p;
}

// GEMM epilogues.
enum { EPI_STORE_F32 = 0, EPI_ADD_F32 = 1, EPI_SWIGLU = 2 };

// bf16 GEMM depth granularity: K (per split) is a multiple of 4 pipeline
// stages of 32.
constexpr int KALIGN = 128;

// Split-K of the residual-adding projections (O and down).  When the live
// row count M leaves too few output tiles to occupy the chip, the GEMM
// splits K into S parts; each writes its raw partial to ws[S][mt*bm][N]
// (mt = row tiles of M) and the next RMSNorm of the residual stream adds
// x += partial_0 + ... + partial_{S-1} (split order) before normalising.
// Both kernels derive S from M with resid_splits, so no host round trip.
struct ResidSplit {
  float* ws;            // NULL: nothing pending
  const int32_t* Mp;    // row count of the producing GEMM
  int nx, bm, K, zmax;  // its column tiles, row tile, depth and largest split
};
constexpr int RESID_TARGET_128 = 256;   // workgroups aimed at with 128-row tiles
constexpr int RESID_TARGET_64 = 512;    // ... with 64-row tiles
__host__ __device__ __forceinline__ int resid_splits(int M, const ResidSplit& r) {
  const int tiles = r.nx * ((M + r.bm - 1) / r.bm);
  const int target = r.bm == 128 ? RESID_TARGET_128 : RESID_TARGET_64;
  int S = 1;
  while (S * 2 <= r.zmax && tiles * S * 2 <= target && r.K % (S * 2 * KALIGN) == 0 &&
         r.K / (S * 2) >= 256)
    S *= 2;
  return S;
}
// Floats of split partials a residual projection of N columns writes for M
// live rows: S(M) whole row-tile slabs of N columns, or 0 when S(M) = 1
// (the add is then done in place).
size_t resid_extent(int M, int N, const ResidSplit& r);
// Largest resid_extent over every live row count M in [1, rows_cap]: the
// workspace a state must hold for that projection.
size_t resid_extent_max(int rows_cap, int N, const ResidSplit& r);

// Quantized projection weights (bf16 models).  fmt WQ_NONE (aux NULL): W
// holds bf16 [N][K].  WQ_FP8: W holds OCP fp8 E4M3 codes [N][K] and aux the
// float power-of-two scale of each row [N].  WQ_MXFP4: W holds E2M1 codes
// stage-major, [K/32][N][16 bytes] (element 2j of a 32-element block in the
// low nibble of byte j, element 2j + 1 in the high nibble), and aux the E8M0
// block exponents [K/32][N] (scale 2^(e - 127)); a matrix of grouped experts
// holds one such block per expert, expert after expert.
enum { WQ_NONE = 0, WQ_FP8 = 1, WQ_MXFP4 = 2 };
struct WQuant {
  int fmt = WQ_NONE;
  const void* aux = nullptr;
};
constexpr int MX_BLOCK = 32;

// ---- launchers (defined in the .hip files) ---------------------------------
// C[M][N] (+)= A[M][K] . W[N][K]^T with M read from *M_dev; grid covers rows_cap.
// bf16 models: A is a bf16 plane pair (hi at A, lo at A + a_plane elements),
// W bf16.  fp32 models: A and W fp32 (a_plane unused).
//   EPI_STORE_F32 / EPI_ADD_F32: out fp32 [M][ldo]
//   EPI_SWIGLU: silu(gate) * up [M][ldo] (W packed gate/up in 16-row groups),
//   as a bf16 plane pair (out_plane) for bf16 models, fp32 otherwise
// wq (bf16 models only): the weight format (WQuant); ldw is W's row stride in
// elements for bf16 and fp8 weights and unused for MXFP4 (N rows per block).
hipError_t launch_gemm(int epi, bool is_bf16, const void* A, int lda, size_t a_plane, const void* W,
                       int ldw, int N, int K, const int32_t* M_dev, int rows_cap, void* out, int ldo,
                       size_t out_plane, hipStream_t st, WQuant wq = WQuant{});
// Expert tiles of a grouped GEMM (all device pointers).
struct GroupTiles {
  const int32_t* tile_e;    // [max_tiles] expert of each tile
  const int32_t* tile_m0;   // [max_tiles] first expert-local row of each tile
  const int32_t* ntiles;    // [1] live tile count
  const int32_t* e_off;     // [E] first expert-sorted row of each expert
  const int32_t* e_cnt;     // [E] rows of each expert
  const int32_t* a_rows;    // optional [assignments] token row of each sorted row
  size_t w_stride;          // weight elements per expert (N x K)
};
constexpr int GROUP_BM = 128;
// out rows are expert-sorted rows; EPI_SWIGLU writes bf16 planes, EPI_STORE_F32 fp32.
// wq: as launch_gemm; fp8 row scales [E][N], MXFP4 codes and exponents one
// stage-major block per expert.
hipError_t launch_gemm_grouped(int epi, const void* A, int lda, size_t a_plane, const void* W,
                               int ldw, int N, int K, const GroupTiles& g, int max_tiles, void* out,
                               int ldo, size_t out_plane, WQuant wq, hipStream_t st);

// MoE routing: softmax over E router logits (fp32 weights [E][d]), top_k
// experts (lowest id among equals), weights renormalised.
hipError_t launch_router(const void* A, size_t a_plane, int d, const float* Wr, int E, int topk,
                         const int32_t* M_dev, int rows_cap, int32_t* top_e, float* top_w,
                         hipStream_t st);
// Deterministic dispatch: expert-sorted assignment lists (token rows ascending
// within each expert), positions of every (row, slot), and the tile list.
struct MoeLists {
  int32_t* e_cnt;    // [E]
  int32_t* e_off;    // [E]
  int32_t* list_row; // [rows_cap * topk]
  int32_t* pos_of;   // [rows_cap * topk]
  int32_t* tile_e;   // [max_tiles]
  int32_t* tile_m0;  // [max_tiles]
  int32_t* ntiles;   // [1]
};
hipError_t launch_moe_dispatch(const int32_t* top_e, int topk, int E, const int32_t* M_dev,
                               const MoeLists& L, hipStream_t st);
// X[row] += sum_j top_w[row][j] * Y[pos_of[row][j]] (fixed slot order).
hipError_t launch_moe_combine(float* X, const float* Y, const int32_t* pos_of, const float* top_w,
                              int topk, int d, const int32_t* M_dev, int rows_cap, hipStream_t st);

struct GemmPlan {
  int bm, bn, zmax;        // tile; largest residual K-split (1 = none)
};
// wide_ok: the 128x256 tile may be chosen (bf16 weights, k_gemm_bf16 kernels)
GemmPlan plan_gemm(bool is_bf16, int N, int K, int rows_cap, bool resid = false, bool wide_ok = false);
// bf16 GEMM with an explicit plan (128x256, 128x128, 64x128 (plain products,
// bf16 weights) or 64x64; K % KALIGN == 0;
// zmax > 1 only for EPI_ADD_F32 with a residual-split workspace ws).
hipError_t launch_gemm_planned(const GemmPlan& p, int epi, const void* A, int lda, size_t a_plane,
                               const void* W, int ldw, int N, int K, const int32_t* M_dev,
                               int rows_cap, void* out, int ldo, size_t out_plane, float* ws,
                               hipStream_t st, WQuant wq = WQuant{});
// Plan of a residual projection (O and down of bf16 models): tile shape and
// the largest K-split (zmax).
GemmPlan plan_resid(int N, int K, int rows_cap, bool wide_ok);
// X[M][N] += A . W^T for the residual stream.  bf16 with a workspace ws of
// ws_floats floats: the kernel may split K (see ResidSplit) and *fold
// describes the pending partials, which the next launch_rmsnorm of X must be
// given; else the add is done in place and fold->ws is NULL.  Returns
// hipErrorInvalidValue, launching nothing, when ws_floats is smaller than
// resid_extent_max of the plan (the partials would not fit).
hipError_t launch_gemm_resid(bool is_bf16, const void* A, int lda, size_t a_plane, const void* W,
                             int ldw, int N, int K, const int32_t* M_dev, int rows_cap, float* X,
                             int ldx, float* ws, size_t ws_floats, ResidSplit* fold, hipStream_t st,
                             WQuant wq = WQuant{});

// LM head: per-row softmax statistics over the vocabulary of
// z = scale * (A . W^T), mask column suppressed.  Writes per-(tile,row)
// partials, then merges them into conf/tok.
hipError_t launch_lm_head(bool is_bf16, const void* A, int d, size_t a_plane, const void* W, int V,
                          int mask_id, float scale, const int32_t* M_dev, int rows_cap,
                          float* part_max, float* part_sum, int32_t* part_arg, float* conf,
                          int32_t* tok, hipStream_t st);
// Debug: full logits [rows][V] for the LM rows (scaled, mask column = -inf).
hipError_t launch_lm_logits(bool is_bf16, const void* A, int d, size_t a_plane, const void* W, int V,
                            int mask_id, float scale, const int32_t* M_dev, int rows_cap,
                            float* logits, hipStream_t st);

// Work item of a workgroup in an XCD-aware launch.  Launches are 1-D with at
// least items + 7 workgroups; the dispatcher deals consecutive workgroups to
// the 8 XCDs in turn, and item u = (id % 8) * ceil(items / 8) + id / 8 gives
// each XCD a contiguous range of items (items are numbered so that neighbours
// share operand tiles), which then stay in that XCD's L2.  Workgroups with
// id >= 8 ceil(items / 8), and those whose u >= items, get u = items (none).
__device__ __forceinline__ int xcd_item(int id, int items) {
  const int per = (items + 7) / 8;
  return id < 8 * per ? (id % 8) * per + id / 8 : items;
}

// Tile (x, y) of work item u in a grid of X column tiles by Y row tiles,
// walked in bands of R row tiles and, inside a band, column by column (the
// band's h <= R row tiles of one column are neighbours).  With the items of
// an XCD-aware launch, the workgroups running at once on one XCD (about 32
// consecutive items of its range) then cover about R row tiles x 32 / R
// column tiles, so each activation row tile and weight column tile they read
// is fetched into that XCD's L2 once for all of them; walking all row tiles
// of a column first would re-fetch the whole activation for every column.
__device__ __forceinline__ void band_tile(int u, int X, int Y, int R, int& x, int& y) {
  const int y0 = (u / (R * X)) * R;
  const int h = Y - y0 < R ? Y - y0 : R;
  const int ub = u - y0 * X;
  x = ub / h;
  y = y0 + ub % h;
}
constexpr int BAND_R = 4;   // row tiles per band: a 128-row hi/lo activation tile is twice a weight tile

// One layer's KV cache.  K: [seq][kv head][pos][hd].  V: bf16 models keep
// it transposed in tiles of 64 keys, [seq][kv head][pos / 64][hd][64]: a
// tile is one contiguous block per plane (DRAM page locality when streamed).
// Inside a tile row, key k sits at slot vt_slot(k): every group of 32 keys is
// reordered so that keys 4j..4j+3 and 16+4j..16+4j+3 fill the 8 adjacent
// slots 8j..8j+7 -- the 8 keys one lane feeds to a P.V MFMA, so that
// fragment is one 16-byte read; aligned runs of 4 keys stay contiguous.
// vt_off gives the offset of (pos, dim) inside a (seq, kv head) slice of
// hd * vstride elements, vstride = maxpos rounded up to 64; vt_row the
// offset of slot 0 of a tile row.  fp32
// models keep V as K.  bf16 models store pairs: lo planes at + k_plane /
// + v_plane elements.  The whole cache is cleared at allocation, so padding
// and not yet written positions are finite.
constexpr int VTILE = 64;
__host__ __device__ __forceinline__ int vt_slot(int k) {
  const int q = k & 31;
  return (k & 32) + 8 * ((q & 15) >> 2) + 4 * (q >> 4) + (q & 3);
}
__host__ __device__ __forceinline__ size_t vt_row(int pos, int dim, int hd) {
  return ((size_t)(pos / VTILE) * hd + dim) * VTILE;
}
__host__ __device__ __forceinline__ size_t vt_off(int pos, int dim, int hd) {
  return vt_row(pos, dim, hd) + vt_slot(pos % VTILE);
}
struct KvView {
  void* K;
  void* V;
  size_t k_plane, v_plane;
  int maxpos, vstride;
};

// Attention of the rows of `plan` over the cache.  bf16 models: tiles of 64
// queries of one (sequence, kv head) (window rows x the q-heads sharing the kv
// head), 64-key tiles staged in LDS; kv_splits > 1 splits every
// query tile's key range into that many workgroups (partials in ws_o
// [splits][rows_cap][H][hd], ws_ml [splits][rows_cap][H][2]) merged in split
// order.  O: bf16 plane pair (lo at O + o_plane elements) for bf16 models,
// fp32 otherwise.
hipError_t launch_attention(bool is_bf16, const void* Q, size_t q_plane, const KvView& kv, void* O,
                            size_t o_plane, PlanView plan, int b, int win_cap, int H, int Hkv,
                            int hd, int B, int kv_splits, float* ws_o, float* ws_ml, int rows_cap,
                            hipStream_t st);
int attention_splits(int b, int win_cap, int rows_est, int H, int Hkv, int hd, int maxpos);

hipError_t launch_embed(bool is_bf16, const int32_t* tokens, int tok_stride, const void* E, int d,
                        int vocab, PlanView plan, int rows_cap, float* X, int32_t* err_flag,
                        hipStream_t st);
// out: fp32 [rows][d] (fp32 models) or a bf16 plane pair (bf16 models,
// lo plane at out + out_plane elements).
// fold: pending residual split partials of the GEMM that produced X (ws
// NULL for none); folded into X (rows reached through gather) first.
hipError_t launch_rmsnorm(bool is_bf16, float* X, const float* g, int d, float eps,
                          const int32_t* M_dev, const int32_t* gather, int rows_cap, void* out,
                          size_t out_plane, const ResidSplit& fold, hipStream_t st);
// fp32 models: RoPE of q and k at the rows' absolute positions; q ->
// Q[row][head][hd], k and v -> the cache (layout of KvView, fp32).
hipError_t launch_rope_kv(const float* QKV, PlanView plan, int rows_cap, int H, int Hkv, int hd,
                          const double* inv_freq, float* Q, const KvView& kv, hipStream_t st);

constexpr int BD_NSTATS = 12;

// Static scratch of the allocation-free decode (bytes per device) and the
// devices it is tracked on.
constexpr size_t BD_STATIC_SCRATCH_BYTES = (size_t)64 << 20;
constexpr int BD_MAX_DEVICES = 64;

struct CommitArgs {
  PlanView in, out;
  const float* conf;        // [lm rows of `in`]
  const int32_t* tok;
  int32_t* tokens;          // [b][tok_stride]
  int tok_stride;           // P + G
  int32_t* commit_step;     // [b][G]
  int32_t* seq_state;       // [b][SS_N]
  int32_t* commit_flag;     // scratch [lm_cap]
  long long* stats;         // [BD_NSTATS] work and participation counters of the executed steps
  int b, P, G, B, nb, mask_id, step;
  float tau;
  int semi_min;             // semi-completion: resolved count that fully activates the next block; -1 = off
  int add_min;              // admission: resolved count of the youngest active block that admits the next
  int skip;                 // static skip rule: leave fully masked blocks behind an active one out
};
hipError_t launch_commit(const CommitArgs& a, hipStream_t st);
// fp8 E4M3 codes of a bf16 matrix [rows][cols], one power-of-two scale per
// row (scale[row] = 2^E, the smallest with max |w| / 2^E <= 448).
hipError_t launch_quant_fp8_rows(const void* W, int rows, int cols, uint8_t* Q, float* scale, hipStream_t st);
// MXFP4 (E2M1 codes, one E8M0 exponent per 32 consecutive elements of a row)
// of a bf16 matrix [rows][cols], cols % 32 == 0, in the stage-major layout of
// WQuant, the rows taken in groups of group_rows (rows % group_rows == 0), each
// group its own block: codes[g][cols/32][group_rows][16], exps[g][cols/32][group_rows].
// Exponent X = floor(log2 max|w|) - 2 over the block (-127 for an all-zero
// block, clamped to [-127, 127]); element code = the E2M1 value nearest to
// w / 2^X, ties to the even mantissa, magnitudes above 6 saturating.
hipError_t launch_quant_mxfp4_rows(const void* W, int rows, int cols, int group_rows, uint8_t* codes,
                                   uint8_t* exps, hipStream_t st);

struct InitArgs {
  PlanView plan;            // step plan to build
  PlanView prefill;         // optional prefill plan to build (hdr NULL = skip)
  int32_t* tokens;          // [b][P + G]
  const int32_t* prompt;    // optional [b][P]: copied into tokens
  int32_t* commit_step;
  int32_t* seq_state;
  int b, P, G, B, nb, mask_id, vocab;
  int add_min;              // as in CommitArgs
  int skip;                 // as in CommitArgs
  int32_t* err_flag;
  long long* stats;         // [BD_NSTATS], cleared
};
hipError_t launch_init_decode(const InitArgs& a, hipStream_t st);

// Debug scatter of per-LM-row conf/tok to [b][G].
hipError_t launch_scatter_stats(const float* conf, const int32_t* tok, PlanView plan, int P, int G,
                                float* dconf, int32_t* dtok, int lm_cap, hipStream_t st);
// QKV projection of bf16 models with RoPE and the cache write in the
// epilogue.  W is the pair-interleaved copy made by launch_permute_qk_rows
// (in each q and k head, packed row 2i = dim i, 2i + 1 = dim i + hd/2, so a
// rotation pair sits in adjacent accumulator lanes); the rotation uses the
// fp64 table of launch_rope_table.  Q -> [rows][H][hd], K and V -> the cache
// (layout of KvView), all as bf16 pairs in the original dimension order.
struct QkvEpi {
  const int32_t* row_seq;   // [rows] plan: sequence of each row
  const int32_t* row_pos;   // [rows] plan: absolute position of each row
  const double* rope;       // [maxpos][hd/2][2]: cos, sin
  void* Q;
  size_t q_plane;
  KvView kv;
  int H, Hkv, hd;
  int rows4;                // 1: every aligned group of 4 rows is 4 consecutive
                            // positions of one sequence (block size % 4 == 0)
};
hipError_t launch_gemm_qkv(const void* A, int lda, size_t a_plane, const void* W, int K,
                           const int32_t* M_dev, int rows_cap, const QkvEpi& e, hipStream_t st,
                           WQuant wq = WQuant{});
// Copy of a [(H + 2 Hkv) hd][d] QKV weight with the q and k head rows
// pair-interleaved (see QkvEpi); v rows unchanged.
hipError_t launch_permute_qk_rows(const void* W, void* out, int H, int Hkv, int hd, size_t row_bytes,
                                  hipStream_t st);
// tab[pos][i] = (cos, sin) of pos * inv_freq[i] in fp64, pos < maxpos, i < hd/2.
hipError_t launch_rope_table(const double* inv_freq, int hd, int maxpos, double* tab, hipStream_t st);

// Interleave gate/up projections in groups of 16 rows (SwiGLU epilogue layout).
hipError_t launch_pack_gate_up(const void* gate, const void* up, void* out, int F, size_t row_bytes,
                               hipStream_t st);

// Zero `bytes` (a multiple of 4) at p (4-byte aligned) with a kernel.
hipError_t launch_zero(void* p, size_t bytes, hipStream_t st);

// Debug scatter of logits rows to [b][G][V].
hipError_t launch_scatter_logits(const float* logits, PlanView plan, int V, int P, int G,
                                 float* out, int lm_cap, hipStream_t st);

}  // namespace bd
