// Host runtime behind the C ABI in include/bd.h: model binding, decode-state
// allocation, and the launch sequence of one denoising step.
//
// One step = embedding gather of the window rows -> per layer {RMSNorm, QKV
// GEMM, RoPE + K/V cache write, block-causal attention, O GEMM + residual,
// RMSNorm, gate/up GEMM with SwiGLU epilogue, down GEMM + residual} -> final
// RMSNorm of the masked rows -> fused LM-head statistics.  Then the commit
// kernel applies the threshold rule, sweeps, admits and writes the next plan.
// Every launch is sized for the largest window and reads the live row counts
// from the device plan, so the host never waits inside a decode.
#include "../../include/bd.h"
#include "bd_internal.h"

#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <mutex>
#include <string>
#include <vector>

using namespace bd;

static thread_local std::string g_err;

static bd_status fail(bd_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define HIPCHK(expr)                                                                      \
  do {                                                                                    \
    hipError_t e_ = (expr);                                                               \
    if (e_ != hipSuccess)                                                                 \
      return fail(BD_EHIP, "%s failed: %s (%s:%d)", #expr, hipGetErrorString(e_), __FILE__, \
                  __LINE__);                                                              \
  } while (0)

struct LayerW {
  const float* attn_norm;
  const void* w_qkv;    // caller's; bf16 models use the pair-interleaved copy w_qkv_p
  void* w_qkv_p;
  const void* w_o;
  const float* ffn_norm;
  void* w_gu;           // dense: packed gate/up (library-owned)
  const void* w_down;
  // MoE
  const float* wr;      // router weights [E][d] (the caller's)
  void* w_gu_e;         // packed gate/up per expert [E][2 Fe][d] (library-owned)
  const void* w_down_e; // [E][d][Fe]
  void* w_gu_s;         // packed shared-expert gate/up [2 Fs][d] (library-owned)
  const void* w_down_s; // [d][Fs]
  // BD_WQ_FP8 / BD_WQ_MXFP4: the projection pointers above hold
  // library-owned codes and these their format and scales (fp8 row scales or
  // MXFP4 block exponents; format WQ_NONE for weights in the model dtype)
  WQuant q_qkv, q_o, q_gu, q_down, q_gu_e, q_down_e, q_gu_s, q_down_s;
};

struct bd_model {
  bd_model_cfg cfg;
  bool bf16;
  size_t esz;
  hipStream_t stream;
  const void* embed;
  std::vector<LayerW> layers;
  const float* final_norm;
  const void* lm_head;
  std::vector<void*> owned;
  double* inv_freq;
  int32_t* err_flag;
  // optional per-kernel-class timing with HIP events on the model's stream
  bool prof = false;
  std::vector<hipEvent_t> ev_pool;
  struct Rec { int kind; hipEvent_t a, b; };
  std::vector<Rec> recs;
  double prof_ms[BD_PROF_KINDS] = {};
  int prof_n[BD_PROF_KINDS] = {};
};

static hipEvent_t take_event(bd_model* m) {
  if (!m->ev_pool.empty()) {
    hipEvent_t e = m->ev_pool.back();
    m->ev_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

struct ProfScope {
  bd_model* m;
  int kind;
  hipEvent_t a = nullptr;
  ProfScope(bd_model* m_, int k) : m(m_), kind(k) {
    if (m->prof && (a = take_event(m))) (void)hipEventRecord(a, m->stream);
  }
  ~ProfScope() {
    if (!a) return;
    hipEvent_t b = take_event(m);
    if (!b) return;
    (void)hipEventRecord(b, m->stream);
    m->recs.push_back({kind, a, b});
  }
};

#define LAUNCH(kind, expr)            \
  do {                                \
    ProfScope ps_(m, (kind));         \
    HIPCHK(expr);                     \
  } while (0)

struct bd_state {
  int b, P, G, B, nb;
  float tau;
  int semi_min, add_min;   // thresholds as resolved counts (see min_resolved)
  int skip;                // static skip rule on
  int maxpos, rows_step, rows_pre, rows_cap, lm_cap, win_step;
  int32_t *tokens, *commit_step, *seq_state, *commit_flag;
  int32_t* plan_buf[3];
  PlanView plan[3];      // [0], [1]: step plans (ping-pong); [2]: prefill
  int cur;
  float* X;
  void* A;
  float* QKV;
  void* Qb;
  void* Ob;
  void* Hact;
  float* resid_ws;         // residual split-K partials (bf16 models)
  size_t resid_ws_floats;
  size_t k_bytes, v_bytes, hact_bytes, act_bytes;   // sizes of the buffers cleared at set-up
  void* Alm;
  float *pmax, *psum;
  int32_t* parg;
  float* conf;
  int32_t* tok;
  float* logits_tmp;
  // bf16 models: plane offsets (elements) of the lo halves of A, Ob, Hact, Alm
  size_t pl_A, pl_O, pl_H, pl_lm;
  int attn_splits;
  float* attn_ws_o;
  float* attn_ws_ml;
  // MoE buffers
  int32_t* top_e;
  float* top_w;
  MoeLists moe;
  int moe_tiles;
  void* act_sorted;      // bf16 plane pair [assign_cap][Fe]
  size_t pl_act;
  float* y_sorted;       // fp32 [assign_cap][d]
  void* Kc;
  void* Vc;
  int vstride;           // V positions per (seq, kv head) slice (bf16: maxpos rounded up to 64)
  double* rope;          // bf16: [maxpos][hd/2] (cos, sin) for the fused QKV epilogue
  int steps;
  bool pending;
  int32_t* host_flag;    // pinned
  long long* stats;      // device [BD_NSTATS]
  std::vector<void*> allocs;
};

static int round_up(int x, int m) { return (x + m - 1) / m * m; }

static bd_status dev_alloc(bd_state* s, void** p, size_t bytes) {
  if (bytes == 0) bytes = 256;
  hipError_t e = hipMalloc(p, bytes);
  if (e != hipSuccess) return fail(BD_ENOMEM, "hipMalloc(%zu) failed: %s", bytes, hipGetErrorString(e));
  s->allocs.push_back(*p);
  return BD_OK;
}

extern "C" const char* bd_last_error(void) { return g_err.c_str(); }

static bd_status scratch_on_current_device(void** out);

namespace bd {
void set_error(const char* msg) { g_err = msg; }
}

// BD_WQ_FP8 / BD_WQ_MXFP4: replace every decoder-layer projection by
// library-owned codes and scales (fp8: one scale per row; MXFP4: one exponent
// per 32 elements of a row, blocks along the input dimension; rows of the
// repacked copies are rows of the original matrices, so the codes do not
// depend on the packing; MoE experts are quantized expert by expert, each a
// stage-major block of its own); the library's bf16 repacked copies are
// released.
static bd_status quantize_layers(bd_model* m) {
  const bd_model_cfg& c = m->cfg;
  const int d = c.d_model, hd = c.head_dim;
  const bool mx = c.wq == BD_WQ_MXFP4;
  std::vector<void*> drop;
  // group_rows: rows of one expert's matrix (MXFP4 stage-major blocks)
  auto q = [&](const void* src, int rows, int cols, int group_rows, bool owned_src, const void** dst,
               WQuant* wq) -> bd_status {
    const size_t n = (size_t)rows * cols;
    uint8_t* codes = nullptr;
    void* aux = nullptr;
    if (hipMalloc((void**)&codes, mx ? n / 2 : n) != hipSuccess) return fail(BD_ENOMEM, "hipMalloc for quantized weights failed");
    m->owned.push_back(codes);
    if (hipMalloc(&aux, mx ? n / MX_BLOCK : (size_t)rows * sizeof(float)) != hipSuccess)
      return fail(BD_ENOMEM, "hipMalloc for weight scales failed");
    m->owned.push_back(aux);
    hipError_t e = mx ? launch_quant_mxfp4_rows(src, rows, cols, group_rows, codes, (uint8_t*)aux, m->stream)
                      : launch_quant_fp8_rows(src, rows, cols, codes, (float*)aux, m->stream);
    if (e != hipSuccess) return fail(BD_EHIP, "weight quantization: %s", hipGetErrorString(e));
    if (owned_src) drop.push_back(const_cast<void*>(src));
    *dst = codes;
    wq->fmt = mx ? WQ_MXFP4 : WQ_FP8;
    wq->aux = aux;
    return BD_OK;
  };
  bd_status r = BD_OK;
  for (LayerW& L : m->layers) {
    const void* p;
    const int nqkv = (c.n_heads + 2 * c.n_kv_heads) * hd;
    if ((r = q(L.w_qkv_p, nqkv, d, nqkv, true, &p, &L.q_qkv)) != BD_OK) return r;
    L.w_qkv_p = const_cast<void*>(p);
    if ((r = q(L.w_o, d, c.n_heads * hd, d, false, &L.w_o, &L.q_o)) != BD_OK) return r;
    if (c.n_experts == 0) {
      if ((r = q(L.w_gu, 2 * c.ffn_dim, d, 2 * c.ffn_dim, true, &p, &L.q_gu)) != BD_OK) return r;
      L.w_gu = const_cast<void*>(p);
      if ((r = q(L.w_down, d, c.ffn_dim, d, false, &L.w_down, &L.q_down)) != BD_OK) return r;
    } else {
      const int E = c.n_experts, Fe = c.expert_ffn, Fs = c.n_shared * c.expert_ffn;
      if ((r = q(L.w_gu_e, E * 2 * Fe, d, 2 * Fe, true, &p, &L.q_gu_e)) != BD_OK) return r;
      L.w_gu_e = const_cast<void*>(p);
      if ((r = q(L.w_down_e, E * d, Fe, d, false, &L.w_down_e, &L.q_down_e)) != BD_OK) return r;
      if (Fs > 0) {
        if ((r = q(L.w_gu_s, 2 * Fs, d, 2 * Fs, true, &p, &L.q_gu_s)) != BD_OK) return r;
        L.w_gu_s = const_cast<void*>(p);
        if ((r = q(L.w_down_s, d, Fs, d, false, &L.w_down_s, &L.q_down_s)) != BD_OK) return r;
      }
    }
  }
  if (hipStreamSynchronize(m->stream) != hipSuccess) return fail(BD_EHIP, "weight quantization failed");
  for (void* p : drop) {
    for (auto it = m->owned.begin(); it != m->owned.end(); ++it)
      if (*it == p) { m->owned.erase(it); break; }
    (void)hipFree(p);
  }
  return BD_OK;
}

extern "C" bd_status bd_quantize_fp8(const void* w, int32_t rows, int32_t cols, uint8_t* codes, float* scale,
                                     void* stream) {
  if (!w || !codes || !scale) return fail(BD_EINVAL, "NULL argument");
  if (rows < 1 || cols < 1) return fail(BD_EINVAL, "need rows, cols >= 1");
  HIPCHK(launch_quant_fp8_rows(w, rows, cols, codes, scale, (hipStream_t)stream));
  return BD_OK;
}

extern "C" bd_status bd_quantize_mxfp4(const void* w, int32_t rows, int32_t cols, int32_t group_rows,
                                       uint8_t* codes, uint8_t* exps, void* stream) {
  if (!w || !codes || !exps) return fail(BD_EINVAL, "NULL argument");
  if (rows < 1 || cols < 1 || group_rows < 1) return fail(BD_EINVAL, "need rows, cols, group_rows >= 1");
  if (cols % MX_BLOCK || rows % group_rows)
    return fail(BD_EINVAL, "cols must be a multiple of 32 and rows of group_rows");
  HIPCHK(launch_quant_mxfp4_rows(w, rows, cols, group_rows, codes, exps, (hipStream_t)stream));
  return BD_OK;
}

extern "C" bd_status bd_init_model(const bd_model_cfg* cfg, const void* const* w, int32_t n_weights,
                                   void* stream, bd_model** out) {
  if (!cfg || !w || !out) return fail(BD_EINVAL, "NULL argument");
  *out = nullptr;
  const bd_model_cfg& c = *cfg;
  if (c.n_layers < 1 || c.d_model < 1 || c.n_heads < 1 || c.n_kv_heads < 1 || c.vocab < 2)
    return fail(BD_EINVAL, "non-positive model dimension");
  if (c.head_dim != 64 && c.head_dim != 128) return fail(BD_EINVAL, "head_dim must be 64 or 128");
  if (c.n_heads % c.n_kv_heads) return fail(BD_EINVAL, "n_heads must be a multiple of n_kv_heads");
  if (c.mask_id < 0 || c.mask_id >= c.vocab) return fail(BD_EINVAL, "mask_id outside [0, vocab)");
  if (c.dtype != BD_F32 && c.dtype != BD_BF16) return fail(BD_EINVAL, "unknown dtype");
  if (c.wq != BD_WQ_NONE && c.wq != BD_WQ_FP8 && c.wq != BD_WQ_MXFP4)
    return fail(BD_EINVAL, "unknown weight precision");
  if (c.wq != BD_WQ_NONE && c.dtype != BD_BF16)
    return fail(BD_EUNSUPPORTED, "fp8 and MXFP4 weights need the bf16 dtype");
  const bool moe = c.n_experts > 0;
  const bool bf16 = c.dtype == BD_BF16;
  const int Fs = moe ? c.n_shared * c.expert_ffn : 0;
  if (moe) {
    if (!bf16) return fail(BD_EUNSUPPORTED, "MoE layers need the bf16 dtype");
    if (c.n_experts > 64 || c.top_k < 1 || c.top_k > c.n_experts || c.expert_ffn < 1 || c.n_shared < 0)
      return fail(BD_EINVAL, "need 1 <= top_k <= n_experts <= 64, expert_ffn >= 1, n_shared >= 0");
    if (c.expert_ffn % 128 || c.d_model % 256)
      return fail(BD_EUNSUPPORTED, "MoE needs expert_ffn a multiple of 128 and d_model of 256");
  } else if (c.ffn_dim < 16 || c.ffn_dim % 16) {
    return fail(BD_EINVAL, "ffn_dim must be a positive multiple of 16");
  }
  const int per_layer = moe ? 11 : 7;
  const int need = 1 + per_layer * c.n_layers + 2;
  if (n_weights != need) return fail(BD_EINVAL, "expected %d weight tensors, got %d", need, n_weights);
  for (int i = 0; i < n_weights; ++i) {
    const int li = (i - 1) % per_layer;
    const bool shared_slot = moe && i >= 1 && i < 1 + per_layer * c.n_layers && li >= 8;
    if (!w[i] && !(shared_slot && Fs == 0)) return fail(BD_EINVAL, "weight %d is NULL", i);
  }
  // GEMM tiling constraints (bf16: N % 128, K % 128; f32: N % 64, K % 16)
  const int nq = bf16 ? 128 : 64, kq = bf16 ? 128 : 16;
  const int qkv = (c.n_heads + 2 * c.n_kv_heads) * c.head_dim;
  const int Fd = moe ? (Fs > 0 ? Fs : 128) : c.ffn_dim;    // width of the dense / shared FFN
  if (qkv % nq || c.d_model % nq || c.vocab % nq || (2 * Fd) % nq || c.d_model % kq ||
      (c.n_heads * c.head_dim) % kq || Fd % kq)
    return fail(BD_EUNSUPPORTED, "dimensions do not fit the GEMM tiles (N %% %d, K %% %d)", nq, kq);

  bd_model* m = new bd_model();
  m->cfg = c;
  m->bf16 = bf16;
  m->esz = bf16 ? 2 : 4;
  m->stream = (hipStream_t)stream;
  int t = 0;
  m->embed = w[t++];
  m->layers.resize(c.n_layers);
  const size_t row_bytes = (size_t)c.d_model * m->esz;
  // library-owned repacked copies (gate/up interleaved for the SwiGLU epilogue)
  auto owned_alloc = [&](size_t bytes) -> void* {
    void* p = nullptr;
    if (hipMalloc(&p, bytes) != hipSuccess) return nullptr;
    m->owned.push_back(p);
    return p;
  };
  auto pack = [&](const void* gate, const void* up, int F, void** out) -> bd_status {
    *out = owned_alloc(2 * (size_t)F * row_bytes);
    if (!*out) return fail(BD_ENOMEM, "hipMalloc for packed gate/up failed");
    hipError_t e = launch_pack_gate_up(gate, up, *out, F, row_bytes, m->stream);
    if (e != hipSuccess) return fail(BD_EHIP, "pack gate/up: %s", hipGetErrorString(e));
    return BD_OK;
  };
  for (int l = 0; l < c.n_layers; ++l) {
    LayerW& L = m->layers[l];
    L = LayerW{};
    L.attn_norm = (const float*)w[t++];
    L.w_qkv = w[t++];
    if (bf16) {
      const int qkv_rows = (c.n_heads + 2 * c.n_kv_heads) * c.head_dim;
      L.w_qkv_p = owned_alloc((size_t)qkv_rows * row_bytes);
      if (!L.w_qkv_p || launch_permute_qk_rows(L.w_qkv, L.w_qkv_p, c.n_heads, c.n_kv_heads, c.head_dim,
                                               row_bytes, m->stream) != hipSuccess) {
        bd_model_free(m);
        return fail(BD_ENOMEM, "QKV weight copy failed");
      }
    }
    L.w_o = w[t++];
    L.ffn_norm = (const float*)w[t++];
    bd_status r = BD_OK;
    if (!moe) {
      const void* gate = w[t++];
      const void* up = w[t++];
      L.w_down = w[t++];
      r = pack(gate, up, c.ffn_dim, &L.w_gu);
    } else {
      const int E = c.n_experts, Fe = c.expert_ffn;
      const float* router = (const float*)w[t++];
      const char* gate_e = (const char*)w[t++];
      const char* up_e = (const char*)w[t++];
      L.w_down_e = w[t++];
      const void* gate_s = w[t++];
      const void* up_s = w[t++];
      L.w_down_s = w[t++];
      L.wr = router;
      {
        L.w_gu_e = owned_alloc((size_t)E * 2 * Fe * row_bytes);
        if (!L.w_gu_e) r = fail(BD_ENOMEM, "hipMalloc for packed experts failed");
        for (int e = 0; e < E && r == BD_OK; ++e) {
          const size_t off = (size_t)e * Fe * row_bytes;
          if (launch_pack_gate_up(gate_e + off, up_e + off, (char*)L.w_gu_e + 2 * off, Fe, row_bytes,
                                  m->stream) != hipSuccess)
            r = fail(BD_EHIP, "pack expert gate/up failed");
        }
      }
      if (r == BD_OK && Fs > 0) r = pack(gate_s, up_s, Fs, &L.w_gu_s);
    }
    if (r != BD_OK) {
      bd_model_free(m);
      return r;
    }
  }
  m->final_norm = (const float*)w[t++];
  m->lm_head = w[t++];
  if (c.wq != BD_WQ_NONE) {
    bd_status r = quantize_layers(m);
    if (r != BD_OK) {
      bd_model_free(m);
      return r;
    }
  }
  std::vector<double> inv(c.head_dim / 2);
  for (int i = 0; i < c.head_dim / 2; ++i)
    inv[i] = pow((double)c.rope_theta, -2.0 * i / (double)c.head_dim);
  hipError_t e1 = hipMalloc((void**)&m->inv_freq, inv.size() * sizeof(double));
  hipError_t e2 = hipMalloc((void**)&m->err_flag, 64);
  if (e1 != hipSuccess || e2 != hipSuccess) {
    bd_model_free(m);
    return fail(BD_ENOMEM, "hipMalloc failed");
  }
  m->owned.push_back(m->inv_freq);
  m->owned.push_back(m->err_flag);
  hipError_t e = hipMemcpyAsync(m->inv_freq, inv.data(), inv.size() * sizeof(double),
                                hipMemcpyHostToDevice, m->stream);
  if (e == hipSuccess) e = hipMemsetAsync(m->err_flag, 0, 64, m->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(m->stream);
  if (e != hipSuccess) {
    bd_model_free(m);
    return fail(BD_EHIP, "model upload: %s", hipGetErrorString(e));
  }
  // device address of the static scratch on this device (bd_decode_static)
  void* scratch_base = nullptr;
  bd_status rs = scratch_on_current_device(&scratch_base);
  if (rs != BD_OK) {
    bd_model_free(m);
    return rs;
  }
  *out = m;
  return BD_OK;
}

extern "C" bd_status bd_model_free(bd_model* m) {
  if (!m) return BD_OK;
  if (m->stream) (void)hipStreamSynchronize(m->stream);
  else (void)hipDeviceSynchronize();
  for (void* p : m->owned) (void)hipFree(p);
  for (auto& r : m->recs) { (void)hipEventDestroy(r.a); (void)hipEventDestroy(r.b); }
  for (hipEvent_t e : m->ev_pool) (void)hipEventDestroy(e);
  delete m;
  return BD_OK;
}

extern "C" bd_status bd_state_free(bd_state* s) {
  if (!s) return BD_OK;
  (void)hipDeviceSynchronize();
  for (void* p : s->allocs) (void)hipFree(p);
  if (s->host_flag) (void)hipHostFree(s->host_flag);
  delete s;
  return BD_OK;
}

// One forward over the rows of `plan`; with `lm` the masked rows get the LM head.
// MoE FFN of one layer (rows of `plan`, operand already in s->A): shared
// expert as a dense SwiGLU FFN added to the residual, router, deterministic
// dispatch, grouped expert GEMMs into expert-sorted buffers, fixed-order
// weighted combine into the residual.
static bd_status run_moe(bd_model* m, bd_state* s, const LayerW& L, const PlanView& plan,
                         int rows_cap) {
  const bd_model_cfg& c = m->cfg;
  const hipStream_t st = m->stream;
  const int d = c.d_model, E = c.n_experts, k = c.top_k, Fe = c.expert_ffn;
  const int Fs = c.n_shared * Fe;
  if (Fs > 0) {
    LAUNCH(BD_PROF_GEMM_GU, launch_gemm(EPI_SWIGLU, true, s->A, d, s->pl_A, L.w_gu_s, d, 2 * Fs, d,
                                        plan.hdr, rows_cap, s->Hact, Fs, s->pl_H, st, L.q_gu_s));
    LAUNCH(BD_PROF_GEMM_DOWN, launch_gemm(EPI_ADD_F32, true, s->Hact, Fs, s->pl_H, L.w_down_s, Fs, d,
                                          Fs, plan.hdr, rows_cap, s->X, d, 0, st, L.q_down_s));
  }
  LAUNCH(BD_PROF_MOE, launch_router(s->A, s->pl_A, d, L.wr, E, k, plan.hdr, rows_cap, s->top_e,
                                    s->top_w, st));
  LAUNCH(BD_PROF_MOE, launch_moe_dispatch(s->top_e, k, E, plan.hdr, s->moe, st));
  GroupTiles g;
  g.tile_e = s->moe.tile_e;
  g.tile_m0 = s->moe.tile_m0;
  g.ntiles = s->moe.ntiles;
  g.e_off = s->moe.e_off;
  g.e_cnt = s->moe.e_cnt;
  g.a_rows = s->moe.list_row;
  g.w_stride = (size_t)2 * Fe * d;
  LAUNCH(BD_PROF_GEMM_GU, launch_gemm_grouped(EPI_SWIGLU, s->A, d, s->pl_A, L.w_gu_e, d, 2 * Fe, d, g,
                                              s->moe_tiles, s->act_sorted, Fe, s->pl_act, L.q_gu_e, st));
  g.a_rows = nullptr;
  g.w_stride = (size_t)d * Fe;
  LAUNCH(BD_PROF_GEMM_DOWN, launch_gemm_grouped(EPI_STORE_F32, s->act_sorted, Fe, s->pl_act,
                                                L.w_down_e, Fe, d, Fe, g, s->moe_tiles, s->y_sorted,
                                                d, 0, L.q_down_e, st));
  LAUNCH(BD_PROF_MOE, launch_moe_combine(s->X, s->y_sorted, s->moe.pos_of, s->top_w, k, d, plan.hdr,
                                         rows_cap, st));
  return BD_OK;
}

static bd_status run_forward(bd_model* m, bd_state* s, const PlanView& plan, int rows_cap,
                             int win_cap, bool lm) {
  const bd_model_cfg& c = m->cfg;
  const bool bf = m->bf16;
  const hipStream_t st = m->stream;
  const int d = c.d_model, H = c.n_heads, Hkv = c.n_kv_heads, hd = c.head_dim, F = c.ffn_dim;
  const int qkv = (H + 2 * Hkv) * hd;
  // cache layout: K [layer][seq][kv head][pos][hd], V [layer][seq][kv head]
  // [vstride / 64][hd][64] (bf16) or as K (fp32); bf16 models keep the lo
  // planes of Q and of each whole cache after the hi planes
  const size_t layer_k = (size_t)s->b * Hkv * s->maxpos * hd;
  const size_t layer_v = (size_t)s->b * Hkv * hd * s->vstride;
  const size_t q_plane = bf ? (size_t)s->rows_cap * H * hd : 0;
  const int kv_splits = (bf && lm) ? s->attn_splits : 1;
  LAUNCH(BD_PROF_EMBED, launch_embed(bf, s->tokens, s->P + s->G, m->embed, d, c.vocab, plan,
                                     rows_cap, s->X, m->err_flag, st));
  ResidSplit pend{};     // residual split partials not yet folded into X
  for (int l = 0; l < c.n_layers; ++l) {
    const LayerW& L = m->layers[l];
    KvView kv;
    kv.K = (char*)s->Kc + l * layer_k * m->esz;
    kv.V = (char*)s->Vc + l * layer_v * m->esz;
    kv.k_plane = bf ? (size_t)c.n_layers * layer_k : 0;
    kv.v_plane = bf ? (size_t)c.n_layers * layer_v : 0;
    kv.maxpos = s->maxpos;
    kv.vstride = s->vstride;
    LAUNCH(BD_PROF_NORM, launch_rmsnorm(bf, s->X, L.attn_norm, d, c.rms_eps, plan.hdr, nullptr,
                                        rows_cap, s->A, s->pl_A, pend, st));
    pend.ws = nullptr;
    if (bf) {
      QkvEpi e;
      e.row_seq = plan.row_seq;
      e.row_pos = plan.row_pos;
      e.rope = s->rope;
      e.Q = s->Qb;
      e.q_plane = q_plane;
      e.kv = kv;
      e.H = H;
      e.Hkv = Hkv;
      e.hd = hd;
      e.rows4 = s->B % 4 == 0;
      LAUNCH(BD_PROF_GEMM_QKV, launch_gemm_qkv(s->A, d, s->pl_A, L.w_qkv_p, d, plan.hdr, rows_cap, e, st,
                                               L.q_qkv));
    } else {
      LAUNCH(BD_PROF_GEMM_QKV, launch_gemm(EPI_STORE_F32, bf, s->A, d, s->pl_A, L.w_qkv, d, qkv, d,
                                           plan.hdr, rows_cap, s->QKV, qkv, 0, st));
      LAUNCH(BD_PROF_ROPE, launch_rope_kv(s->QKV, plan, rows_cap, H, Hkv, hd, m->inv_freq,
                                          (float*)s->Qb, kv, st));
    }
    LAUNCH(BD_PROF_ATTN, launch_attention(bf, s->Qb, q_plane, kv,
                                          s->Ob, s->pl_O, plan, s->b, win_cap, H, Hkv, hd, s->B,
                                          kv_splits, s->attn_ws_o, s->attn_ws_ml, rows_cap, st));
    LAUNCH(BD_PROF_GEMM_O, launch_gemm_resid(bf, s->Ob, H * hd, s->pl_O, L.w_o, H * hd, d, H * hd,
                                             plan.hdr, rows_cap, s->X, d, s->resid_ws, s->resid_ws_floats, &pend, st,
                                             L.q_o));
    LAUNCH(BD_PROF_NORM, launch_rmsnorm(bf, s->X, L.ffn_norm, d, c.rms_eps, plan.hdr, nullptr,
                                        rows_cap, s->A, s->pl_A, pend, st));
    pend.ws = nullptr;
    if (c.n_experts == 0) {
      LAUNCH(BD_PROF_GEMM_GU, launch_gemm(EPI_SWIGLU, bf, s->A, d, s->pl_A, L.w_gu, d, 2 * F, d,
                                          plan.hdr, rows_cap, s->Hact, F, s->pl_H, st, L.q_gu));
      LAUNCH(BD_PROF_GEMM_DOWN, launch_gemm_resid(bf, s->Hact, F, s->pl_H, L.w_down, F, d, F,
                                                  plan.hdr, rows_cap, s->X, d, s->resid_ws, s->resid_ws_floats, &pend,
                                                  st, L.q_down));
    } else {
      bd_status r = run_moe(m, s, L, plan, rows_cap);
      if (r != BD_OK) return r;
    }
  }
  if (lm) {
    LAUNCH(BD_PROF_NORM, launch_rmsnorm(bf, s->X, m->final_norm, d, c.rms_eps, plan.hdr + 1,
                                        plan.lm_row, s->lm_cap, s->Alm, s->pl_lm, pend, st));
    LAUNCH(BD_PROF_LM_HEAD, launch_lm_head(bf, s->Alm, d, s->pl_lm, m->lm_head, c.vocab, c.mask_id,
                                           c.logit_scale, plan.hdr + 1, s->lm_cap, s->pmax, s->psum,
                                           s->parg, s->conf, s->tok, st));
  }
  return BD_OK;
}

static bd_status check_err_flag(bd_model* m) {
  int32_t flag = 0;
  HIPCHK(hipMemcpyAsync(&flag, m->err_flag, sizeof flag, hipMemcpyDeviceToHost, m->stream));
  HIPCHK(hipStreamSynchronize(m->stream));
  if (flag) {
    HIPCHK(hipMemsetAsync(m->err_flag, 0, sizeof flag, m->stream));
    return fail(BD_EINVAL, "token id outside [0, vocab) in a prompt");
  }
  return BD_OK;
}

// Smallest resolved count r in [0, B] whose float32 fraction r / B reaches
// thr (float32 compare), or B + 1 when none does.
static int min_resolved(float thr, int B) {
  for (int r = 0; r <= B; ++r)
    if ((float)r / (float)B >= thr) return r;
  return B + 1;
}

// Floats of residual split partials the O and down projections of a bf16
// model may write over rows_cap rows (the largest of the two extents; they
// never hold partials at the same time: the RMSNorm between them folds them).
static ResidSplit resid_split_of(int N, int K, int rows_cap, bool wide_ok = true) {
  const GemmPlan p = plan_resid(N, K, rows_cap, wide_ok);
  ResidSplit r{};
  r.nx = N / p.bn;
  r.bm = p.bm;
  r.K = K;
  r.zmax = p.zmax;
  return r;
}

static size_t resid_ws_need(const bd_model_cfg& c, int rows_cap) {
  // the larger extent of the bf16-weight and the quantized-weight plans
  const int d = c.d_model;
  size_t need = 0;
  for (int wide = 0; wide < 2; ++wide) {
    const size_t o = resid_extent_max(rows_cap, d, resid_split_of(d, c.n_heads * c.head_dim, rows_cap, wide));
    if (o > need) need = o;
    if (c.n_experts == 0) {
      const size_t dn = resid_extent_max(rows_cap, d, resid_split_of(d, c.ffn_dim, rows_cap, wide));
      if (dn > need) need = dn;
    }
  }
  return need;
}

extern "C" bd_status bd_plan_projection(int32_t N, int32_t K, int32_t rows_cap, int32_t resid,
                                        int32_t* bm_out, int32_t* bn_out, int32_t* zmax_out,
                                        int64_t* ws_floats_out) {
  if (N < 1 || K < 1 || rows_cap < 1) return fail(BD_EINVAL, "need N, K, rows_cap >= 1");
  if (N % 128 || K % KALIGN) return fail(BD_EUNSUPPORTED, "N and K must be multiples of 128");
  GemmPlan p;
  int64_t wsf = 0;
  if (resid) {
    p = plan_resid(N, K, rows_cap, true);
    wsf = (int64_t)resid_extent_max(rows_cap, N, resid_split_of(N, K, rows_cap));
  } else {
    p = plan_gemm(true, N, K, rows_cap, false, true);
  }
  if (bm_out) *bm_out = p.bm;
  if (bn_out) *bn_out = p.bn;
  if (zmax_out) *zmax_out = p.zmax;
  if (ws_floats_out) *ws_floats_out = wsf;
  return BD_OK;
}

// Where a state's device buffers come from.  HEAP: one hipMalloc per buffer
// (owned by the state, released by bd_state_free).  COUNT: nothing is
// allocated, only the bytes the layout needs are summed.  CARVE: consecutive
// 256-byte-aligned slices of a region the caller provides (nothing is
// allocated; the region must hold the COUNT total).
struct Arena {
  enum Mode { HEAP, COUNT, CARVE } mode = HEAP;
  char* base = nullptr;
  size_t cap = 0, used = 0;
};

static bd_status arena_alloc(bd_state* s, Arena& ar, void** p, size_t bytes) {
  if (bytes == 0) bytes = 256;
  const size_t sz = (bytes + 255) & ~(size_t)255;
  if (ar.mode == Arena::HEAP) return dev_alloc(s, p, bytes);
  if (ar.mode == Arena::COUNT) {
    *p = nullptr;
    ar.used += sz;
    return BD_OK;
  }
  if (ar.used + sz > ar.cap) return fail(BD_ENOMEM, "state needs more than %zu bytes of scratch", ar.cap);
  *p = ar.base + ar.used;
  ar.used += sz;
  return BD_OK;
}

static bd_status check_decode_args(const bd_model* m, const int32_t* prompt, int32_t b, int32_t P, int32_t G,
                                   const bd_decode_cfg* cfg) {
  if (!m || !cfg) return fail(BD_EINVAL, "NULL argument");
  const int B = cfg->block_size, nb = cfg->n_inflight;
  if (b < 1 || P < 0 || G < 1 || B < 1 || nb < 1) return fail(BD_EINVAL, "need b, G, B, n_inflight >= 1 and P >= 0");
  if (P % B || G % B) return fail(BD_EINVAL, "P and G must be multiples of the block size");
  if (isnan(cfg->tau) || isnan(cfg->tau_semi) || isnan(cfg->tau_add))
    return fail(BD_EINVAL, "tau, tau_semi or tau_add is NaN");
  if (cfg->skip_masked != 0 && cfg->skip_masked != 1) return fail(BD_EINVAL, "skip_masked must be 0 or 1");
  if (P > 0 && !prompt) return fail(BD_EINVAL, "NULL prompt");
  if (b > 256) return fail(BD_EUNSUPPORTED, "at most 256 sequences per state");
  if (nb > 8) return fail(BD_EUNSUPPORTED, "at most 8 in-flight blocks");
  return BD_OK;
}

// Sizes of the state and its device buffers, taken from the arena (no
// device work).
static bd_status state_layout(const bd_model* m, int32_t b, int32_t P, int32_t G, const bd_decode_cfg* cfg,
                              bd_state* s, Arena& ar) {
  const bd_model_cfg& c = m->cfg;
  const int B = cfg->block_size, nb = cfg->n_inflight;
  s->b = b; s->P = P; s->G = G; s->B = B; s->nb = nb; s->tau = cfg->tau;
  s->semi_min = cfg->tau_semi < 0.0f ? -1 : min_resolved(cfg->tau_semi, B);
  s->add_min = min_resolved(cfg->tau_add, B);
  s->skip = cfg->skip_masked;
  s->maxpos = P + G;
  s->win_step = 2 * nb * B;
  s->rows_step = round_up(b * s->win_step, 256);
  s->rows_pre = round_up(b * P, 256);
  s->rows_cap = s->rows_step > s->rows_pre ? s->rows_step : s->rows_pre;
  s->lm_cap = round_up(b * nb * B, 256);
  const int d = c.d_model, H = c.n_heads, Hkv = c.n_kv_heads, hd = c.head_dim;
  const int qkv = (H + 2 * Hkv) * hd;
  const int ntiles = c.vocab / (m->bf16 ? 128 : 64);
  // the expert gate/up product gathers its token rows by 32-bit byte
  // offsets from the start of an activation plane
  if (c.n_experts > 0 && m->bf16 && (size_t)s->rows_cap * d * 2 >= ((size_t)1 << 32))
    return fail(BD_EUNSUPPORTED, "MoE activation plane of %zu bytes: at most 4 GiB (fewer sequences or a shorter prompt)",
                (size_t)s->rows_cap * d * 2);
  bd_status r = BD_OK;
#define ALLOC(ptr, bytes)                                                  \
  do {                                                                     \
    if ((r = arena_alloc(s, ar, (void**)&(ptr), (bytes))) != BD_OK) return r; \
  } while (0)
  ALLOC(s->tokens, (size_t)b * (P + G) * 4);
  ALLOC(s->commit_step, (size_t)b * G * 4);
  ALLOC(s->seq_state, (size_t)b * SS_N * 4);
  ALLOC(s->stats, BD_NSTATS * sizeof(long long));
  ALLOC(s->commit_flag, (size_t)s->lm_cap * 4);
  for (int i = 0; i < 3; ++i) {
    const int rc = i < 2 ? s->rows_step : s->rows_pre;
    ALLOC(s->plan_buf[i], plan_words(rc, s->lm_cap, b) * 4);
    s->plan[i] = plan_view(s->plan_buf[i], rc, s->lm_cap, b);
  }
  ALLOC(s->X, (size_t)s->rows_cap * d * 4);
  // activation operands: fp32, or two bf16 planes (same bytes) for bf16 models
  ALLOC(s->A, (size_t)s->rows_cap * d * 4);
  if (m->bf16) {
    s->pl_A = (size_t)s->rows_cap * d;
    s->pl_O = (size_t)s->rows_cap * H * hd;
    s->pl_H = (size_t)s->rows_cap * (c.n_experts ? c.n_shared * c.expert_ffn : c.ffn_dim);
    s->pl_lm = (size_t)s->lm_cap * d;
  }
  if (!m->bf16) ALLOC(s->QKV, (size_t)s->rows_cap * qkv * 4);
  ALLOC(s->Qb, (size_t)s->rows_cap * H * hd * 4);     // fp32, or a bf16 plane pair
  ALLOC(s->Ob, (size_t)s->rows_cap * H * hd * 4);
  const int Fh = c.n_experts ? c.n_shared * c.expert_ffn : c.ffn_dim;   // dense / shared FFN width
  s->hact_bytes = (size_t)s->rows_cap * (Fh > 0 ? Fh : 1) * 4;
  ALLOC(s->Hact, s->hact_bytes);
  ALLOC(s->Alm, (size_t)s->lm_cap * d * 4);
  ALLOC(s->pmax, (size_t)ntiles * s->lm_cap * 4);
  ALLOC(s->psum, (size_t)ntiles * s->lm_cap * 4);
  ALLOC(s->parg, (size_t)ntiles * s->lm_cap * 4);
  ALLOC(s->conf, (size_t)s->lm_cap * 4);
  ALLOC(s->tok, (size_t)s->lm_cap * 4);
  // fp32 values or 2 bf16 planes: 4 bytes per element either way
  s->vstride = m->bf16 ? round_up(s->maxpos, 64) : s->maxpos;
  s->k_bytes = (size_t)c.n_layers * b * Hkv * s->maxpos * hd * 4;
  s->v_bytes = (size_t)c.n_layers * b * Hkv * hd * s->vstride * 4;
  ALLOC(s->Kc, s->k_bytes);
  ALLOC(s->Vc, s->v_bytes);
  if (m->bf16) ALLOC(s->rope, (size_t)s->maxpos * hd * sizeof(double));
  if (m->bf16) {
    s->resid_ws_floats = resid_ws_need(c, s->rows_step);
    const size_t pre = resid_ws_need(c, s->rows_pre);
    if (pre > s->resid_ws_floats) s->resid_ws_floats = pre;
    // a small workspace even when K is never split keeps the residual tile plan
    if (s->resid_ws_floats < 64) s->resid_ws_floats = 64;
    ALLOC(s->resid_ws, s->resid_ws_floats * sizeof(float));
  }
  if (c.n_experts > 0) {
    const int E = c.n_experts, k = c.top_k, Fe = c.expert_ffn;
    const size_t assign_cap = (size_t)s->rows_cap * k + GROUP_BM;   // + one tile of padding rows
    s->moe_tiles = (int)((size_t)s->rows_cap * k / GROUP_BM) + E + 1;
    ALLOC(s->top_e, (size_t)s->rows_cap * k * 4);
    ALLOC(s->top_w, (size_t)s->rows_cap * k * 4);
    ALLOC(s->moe.e_cnt, (size_t)E * 4);
    ALLOC(s->moe.e_off, (size_t)E * 4);
    ALLOC(s->moe.list_row, assign_cap * 4);
    ALLOC(s->moe.pos_of, (size_t)s->rows_cap * k * 4);
    ALLOC(s->moe.tile_e, (size_t)s->moe_tiles * 4);
    ALLOC(s->moe.tile_m0, (size_t)s->moe_tiles * 4);
    ALLOC(s->moe.ntiles, 16);
    s->act_bytes = assign_cap * Fe * 4;
    ALLOC(s->act_sorted, s->act_bytes);
    s->pl_act = assign_cap * Fe;
    ALLOC(s->y_sorted, assign_cap * d * 4);
  }
  s->attn_splits = m->bf16 ? attention_splits(b, s->win_step, nb * B, H, Hkv, hd, s->maxpos) : 1;
  if (s->attn_splits > 1) {
    ALLOC(s->attn_ws_o, (size_t)s->attn_splits * s->rows_step * H * hd * 4);
    ALLOC(s->attn_ws_ml, (size_t)s->attn_splits * s->rows_step * H * 2 * 4);
  }
#undef ALLOC
  return BD_OK;
}

// Device-side set-up of a laid-out state: RoPE table, cleared buffers, the
// first plan and the prompt's forward.  Asynchronous, on the model's stream.
static bd_status state_init(bd_model* m, const int32_t* prompt, bd_state* s) {
  const bd_model_cfg& c = m->cfg;
  const hipStream_t st = m->stream;
  const int d = c.d_model, H = c.n_heads, hd = c.head_dim;
  if (m->bf16) HIPCHK(launch_rope_table(m->inv_freq, hd, s->maxpos, s->rope, st));
  // Row buffers are read in whole GEMM tiles: clear them once so that rows
  // past the live count never hold NaN patterns.  The caches are cleared too:
  // attention tiles read (and weigh by zero) positions past the live keys.
  HIPCHK(launch_zero(s->A, (size_t)s->rows_cap * d * 4, st));
  HIPCHK(launch_zero(s->Kc, s->k_bytes, st));
  HIPCHK(launch_zero(s->Vc, s->v_bytes, st));
  HIPCHK(launch_zero(s->Ob, (size_t)s->rows_cap * H * hd * 4, st));
  HIPCHK(launch_zero(s->Hact, s->hact_bytes, st));
  HIPCHK(launch_zero(s->Alm, (size_t)s->lm_cap * d * 4, st));
  if (c.n_experts > 0) HIPCHK(launch_zero(s->act_sorted, s->act_bytes, st));
  InitArgs ia;
  ia.plan = s->plan[0];
  ia.prefill = s->plan[2];
  ia.tokens = s->tokens;
  ia.prompt = s->P > 0 ? prompt : nullptr;
  ia.commit_step = s->commit_step;
  ia.seq_state = s->seq_state;
  ia.b = s->b; ia.P = s->P; ia.G = s->G; ia.B = s->B; ia.nb = s->nb; ia.mask_id = c.mask_id;
  ia.vocab = c.vocab;
  ia.add_min = s->add_min;
  ia.skip = s->skip;
  ia.err_flag = m->err_flag;
  ia.stats = s->stats;
  HIPCHK(launch_init_decode(ia, st));
  s->cur = 0;
  s->steps = 0;
  s->pending = false;
  if (s->P > 0) return run_forward(m, s, s->plan[2], s->rows_pre, s->P, false);
  return BD_OK;
}

extern "C" bd_status bd_prefill(bd_model* m, const int32_t* prompt, int32_t b, int32_t P, int32_t G,
                                const bd_decode_cfg* cfg, bd_state** out) {
  if (!out) return fail(BD_EINVAL, "NULL argument");
  *out = nullptr;
  bd_status r = check_decode_args(m, prompt, b, P, G, cfg);
  if (r != BD_OK) return r;
  bd_state* s = new bd_state();
  Arena heap;
  if ((r = state_layout(m, b, P, G, cfg, s, heap)) != BD_OK) {
    bd_state_free(s);
    return r;
  }
  if (hipHostMalloc((void**)&s->host_flag, 64, hipHostMallocDefault) != hipSuccess) {
    s->host_flag = nullptr;
    bd_state_free(s);
    return fail(BD_ENOMEM, "hipHostMalloc failed");
  }
  if ((r = state_init(m, prompt, s)) != BD_OK) {
    bd_state_free(s);
    return r;
  }
  *out = s;
  return BD_OK;
}

extern "C" bd_status bd_state_reset(bd_model* m, bd_state* s) {
  if (!m || !s) return fail(BD_EINVAL, "NULL argument");
  InitArgs ia;
  ia.plan = s->plan[0];
  ia.prefill = PlanView{};
  ia.prefill.hdr = nullptr;
  ia.tokens = s->tokens;
  ia.prompt = nullptr;
  ia.commit_step = s->commit_step;
  ia.seq_state = s->seq_state;
  ia.b = s->b; ia.P = s->P; ia.G = s->G; ia.B = s->B; ia.nb = s->nb; ia.add_min = s->add_min;
  ia.skip = s->skip;
  ia.mask_id = m->cfg.mask_id; ia.vocab = m->cfg.vocab; ia.err_flag = m->err_flag;
  ia.stats = s->stats;
  HIPCHK(launch_init_decode(ia, m->stream));
  s->cur = 0;
  s->steps = 0;
  s->pending = false;
  return BD_OK;
}

extern "C" bd_status bd_state_steps(const bd_state* s, int32_t* out) {
  if (!s || !out) return fail(BD_EINVAL, "NULL argument");
  *out = s->steps;
  return BD_OK;
}

extern "C" bd_status bd_denoise_step(bd_model* m, bd_state* s, float* conf_dev, int32_t* tok_dev,
                                     float* logits_dev) {
  if (!m || !s) return fail(BD_EINVAL, "NULL argument");
  if (s->pending) return fail(BD_ESTATE, "previous step not committed");
  const PlanView& plan = s->plan[s->cur];
  bd_status r = run_forward(m, s, plan, s->rows_step, s->win_step, true);
  if (r != BD_OK) return r;
  const bd_model_cfg& c = m->cfg;
  if (conf_dev || tok_dev)
    HIPCHK(launch_scatter_stats(s->conf, s->tok, plan, s->P, s->G, conf_dev, tok_dev, s->lm_cap,
                                m->stream));
  if (logits_dev) {
    if (!s->logits_tmp) {
      if ((r = dev_alloc(s, (void**)&s->logits_tmp, (size_t)s->lm_cap * c.vocab * 4)) != BD_OK) return r;
    }
    HIPCHK(launch_lm_logits(m->bf16, s->Alm, c.d_model, s->pl_lm, m->lm_head, c.vocab, c.mask_id, c.logit_scale,
                            plan.hdr + 1, s->lm_cap, s->logits_tmp, m->stream));
    HIPCHK(launch_scatter_logits(s->logits_tmp, plan, c.vocab, s->P, s->G, logits_dev, s->lm_cap,
                                 m->stream));
  }
  s->pending = true;
  return BD_OK;
}

extern "C" bd_status bd_commit(bd_model* m, bd_state* s, int32_t* all_done_host) {
  if (!m || !s) return fail(BD_EINVAL, "NULL argument");
  if (!s->pending) return fail(BD_ESTATE, "no denoising step to commit");
  CommitArgs a;
  a.in = s->plan[s->cur];
  a.out = s->plan[s->cur ^ 1];
  a.conf = s->conf;
  a.tok = s->tok;
  a.tokens = s->tokens;
  a.tok_stride = s->P + s->G;
  a.commit_step = s->commit_step;
  a.seq_state = s->seq_state;
  a.commit_flag = s->commit_flag;
  a.b = s->b; a.P = s->P; a.G = s->G; a.B = s->B; a.nb = s->nb;
  a.mask_id = m->cfg.mask_id;
  a.step = s->steps;
  a.tau = s->tau;
  a.semi_min = s->semi_min;
  a.add_min = s->add_min;
  a.skip = s->skip;
  a.stats = s->stats;
  LAUNCH(BD_PROF_COMMIT, launch_commit(a, m->stream));
  s->cur ^= 1;
  s->steps += 1;
  s->pending = false;
  if (all_done_host) {
    int32_t flag = 0;     // states in the static scratch have no pinned flag
    int32_t* dst = s->host_flag ? s->host_flag : &flag;
    HIPCHK(hipMemcpyAsync(dst, s->plan[s->cur].hdr + 2, 4, hipMemcpyDeviceToHost, m->stream));
    HIPCHK(hipStreamSynchronize(m->stream));
    *all_done_host = *dst;
    bd_status r = check_err_flag(m);
    if (r != BD_OK) return r;
  }
  return BD_OK;
}

__global__ void k_read_trace(const int32_t* __restrict__ tokens, const int32_t* __restrict__ cs,
                             const int32_t* __restrict__ ss, int b, int P, int G,
                             int32_t* __restrict__ t_out, int32_t* __restrict__ c_out,
                             int32_t* __restrict__ f_out) {
  const int s = blockIdx.x;
  for (int j = threadIdx.x; j < G; j += blockDim.x) {
    if (t_out) t_out[(size_t)s * G + j] = tokens[(size_t)s * (P + G) + P + j];
    if (c_out) c_out[(size_t)s * G + j] = cs[(size_t)s * G + j];
  }
  if (f_out && threadIdx.x == 0) f_out[s] = ss[s * SS_N + SS_FORWARDS];
}

extern "C" bd_status bd_state_read(bd_model* m, bd_state* s, int32_t* tokens_dev,
                                   int32_t* commit_step_dev, int32_t* forwards_dev) {
  if (!m || !s) return fail(BD_EINVAL, "NULL argument");
  k_read_trace<<<s->b, 256, 0, m->stream>>>(s->tokens, s->commit_step, s->seq_state, s->b, s->P, s->G,
                                            tokens_dev, commit_step_dev, forwards_dev);
  HIPCHK(hipGetLastError());
  HIPCHK(hipStreamSynchronize(m->stream));
  return check_err_flag(m);
}

// Denoising steps until every sequence is done.  Each step commits at least
// one token of every unfinished sequence, so G steps always suffice; the
// host checks the device flag every few steps (steps after completion are
// empty launches).
static bd_status run_decode_loop(bd_model* m, bd_state* s) {
  const int check = 4;
  int32_t done = 0;
  bd_status r = BD_OK;
  while (!done) {
    for (int k = 0; k < check && r == BD_OK; ++k) {
      r = bd_denoise_step(m, s, nullptr, nullptr, nullptr);
      if (r == BD_OK) r = bd_commit(m, s, (k == check - 1) ? &done : nullptr);
    }
    if (r != BD_OK) return r;
    if (!done && s->steps > s->G + check) return fail(BD_ESTATE, "decode did not finish within %d steps", s->steps);
  }
  return BD_OK;
}

extern "C" bd_status bd_decode(bd_model* m, const int32_t* prompt, int32_t b, int32_t P, int32_t G,
                               const bd_decode_cfg* cfg, int32_t* tokens_dev, int32_t* commit_step_dev,
                               int32_t* forwards_dev) {
  bd_state* s = nullptr;
  bd_status r = bd_prefill(m, prompt, b, P, G, cfg, &s);
  if (r != BD_OK) return r;
  r = run_decode_loop(m, s);
  if (r == BD_OK) r = bd_state_read(m, s, tokens_dev, commit_step_dev, forwards_dev);
  bd_state_free(s);
  return r;
}

// ---- decode without allocation ---------------------------------------------
// The static scratch that bd_decode_static lays its state out in.  Each
// device holds its own copy from the library's load until the process ends.
// In host code `scratch` only stands for the symbol: its device address on
// each device comes from hipGetSymbolAddress (looked up once per device, at
// bd_init_model or at the first call on the device) and only that address is
// handed to kernels.
static_assert(BD_STATIC_SCRATCH_BYTES == BD_STATIC_SCRATCH_BYTES_VALUE, "scratch size as declared in bd.h");
static __device__ __align__(256) unsigned char scratch[BD_STATIC_SCRATCH_BYTES];
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[BD_MAX_DEVICES];

static bd_status scratch_on_current_device(void** out) {
  int dev = -1;
  HIPCHK(hipGetDevice(&dev));
  if (dev < 0 || dev >= BD_MAX_DEVICES) return fail(BD_EUNSUPPORTED, "device %d outside [0, %d)", dev, BD_MAX_DEVICES);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return fail(BD_EHIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return BD_OK;
}

extern "C" bd_status bd_decode_static(bd_model* m, const int32_t* prompt, int32_t b, int32_t P, int32_t G,
                                      const bd_decode_cfg* cfg, int32_t* tokens_dev, int32_t* commit_step_dev,
                                      int32_t* forwards_dev) {
  bd_status r = check_decode_args(m, prompt, b, P, G, cfg);
  if (r != BD_OK) return r;
  bd_state s{};
  Arena count;
  count.mode = Arena::COUNT;
  if ((r = state_layout(m, b, P, G, cfg, &s, count)) != BD_OK) return r;
  if (count.used > BD_STATIC_SCRATCH_BYTES)
    return fail(BD_EUNSUPPORTED, "this decode needs %zu bytes of state; the static scratch holds %zu "
                "(use bd_decode)", count.used, (size_t)BD_STATIC_SCRATCH_BYTES);
  void* base = nullptr;
  if ((r = scratch_on_current_device(&base)) != BD_OK) return r;
  Arena carve;
  carve.mode = Arena::CARVE;
  carve.base = (char*)base;
  carve.cap = BD_STATIC_SCRATCH_BYTES;
  bd_state t{};
  if ((r = state_layout(m, b, P, G, cfg, &t, carve)) != BD_OK) return r;
  const bool prof = m->prof;     // per-launch timing would create events: off for this call
  m->prof = false;
  r = state_init(m, prompt, &t);
  if (r == BD_OK) r = run_decode_loop(m, &t);
  if (r == BD_OK) r = bd_state_read(m, &t, tokens_dev, commit_step_dev, forwards_dev);
  else (void)hipStreamSynchronize(m->stream);   // leave no work in flight on the scratch
  m->prof = prof;
  return r;
}

extern "C" bd_status bd_state_stats(bd_model* m, bd_state* s, int64_t* out, int32_t n) {
  if (!m || !s || !out || n < 1 || n > BD_NSTATS) return fail(BD_EINVAL, "bad arguments");
  long long tmp[BD_NSTATS];
  HIPCHK(hipMemcpyAsync(tmp, s->stats, sizeof tmp, hipMemcpyDeviceToHost, m->stream));
  HIPCHK(hipStreamSynchronize(m->stream));
  for (int i = 0; i < n; ++i) out[i] = (int64_t)tmp[i];
  return BD_OK;
}

extern "C" bd_status bd_profile(bd_model* m, int32_t enable) {
  if (!m) return fail(BD_EINVAL, "NULL model");
  HIPCHK(hipStreamSynchronize(m->stream));
  for (auto& r : m->recs) { m->ev_pool.push_back(r.a); m->ev_pool.push_back(r.b); }
  m->recs.clear();
  for (int k = 0; k < BD_PROF_KINDS; ++k) { m->prof_ms[k] = 0.0; m->prof_n[k] = 0; }
  m->prof = enable != 0;
  return BD_OK;
}

extern "C" bd_status bd_profile_read(bd_model* m, double* ms_out, int32_t* count_out) {
  if (!m) return fail(BD_EINVAL, "NULL model");
  HIPCHK(hipStreamSynchronize(m->stream));
  for (auto& r : m->recs) {
    float ms = 0.f;
    HIPCHK(hipEventElapsedTime(&ms, r.a, r.b));
    m->prof_ms[r.kind] += ms;
    m->prof_n[r.kind] += 1;
    m->ev_pool.push_back(r.a);
    m->ev_pool.push_back(r.b);
  }
  m->recs.clear();
  for (int k = 0; k < BD_PROF_KINDS; ++k) {
    if (ms_out) ms_out[k] = m->prof_ms[k];
    if (count_out) count_out[k] = m->prof_n[k];
  }
  return BD_OK;
}
