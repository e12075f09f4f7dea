// Host runtime and C ABI of the DFlare draft step (see include/dflare.h).
//
// One handle owns: the re-packed weights, the cached fusion weights alpha, the
// per-draft-layer context cache (K as [n_kv, Lcap, hd], V transposed as
// [n_kv, hd, Lcap], both bf16), a rotary table, and the scratch of one step.
// Every call enqueues a fixed sequence of kernels on the handle's stream; the
// values that change between calls (L, n_new, positions) travel through a
// device-resident StepParams block written by a one-thread prologue kernel.
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <unordered_set>
#include <vector>

#include "dflare.h"
#include "dflare_impl.h"

using namespace dflare;

namespace {

const uint32_t kMagic = 0xDF1A2E00u;

struct Plan {
  int nt = 4;      // output tiles per block
  int waves = 4;   // waves per block (they split K)
  int groups = 1;  // blocks per layer and row tile
};

std::mutex g_mu;
std::unordered_set<const dflare_handle*> g_live;
thread_local std::string g_init_error;

int ceil_div(long a, long b) { return (int)((a + b - 1) / b); }

}  // namespace

struct dflare_handle {
  uint32_t magic = kMagic;
  dflare_config cfg{};
  hipStream_t stream = nullptr;
  int L = 0;
  int Lcap = 0;
  int q_dim = 0, kv_dim = 0;
  int Rpad = 0;
  // packed weights
  u32x4 *w_qkv = nullptr, *w_o = nullptr, *w_gu = nullptr, *w_down = nullptr, *w_kvt = nullptr, *w_lm = nullptr;
  long s_qkv = 0, s_o = 0, s_gu = 0, s_down = 0, s_kvt = 0;
  uint16_t* embed = nullptr;
  float *g_fuse = nullptr, *g_attn = nullptr, *g_mlp = nullptr, *g_final = nullptr;
  float* alpha = nullptr;
  std::vector<float> alpha_host;
  // context cache
  uint16_t *kc = nullptr, *vt = nullptr;
  long cache_layer_stride = 0;
  long cache_plane = 0;
  float2* rope = nullptr;
  // step scratch
  StepParams* params = nullptr;
  int* ids = nullptr;
  float *X = nullptr, *Xstats = nullptr, *Q = nullptr;
  float* Ustats = nullptr;
  // activations in A-fragment layout (hi / lo bf16 planes), each padded by 64 tiles
  u32x4 *xa_hi = nullptr, *xa_lo = nullptr;  // x * gain of the next RMSNorm consumer, [Kt_H]
  u32x4 *oa_hi = nullptr, *oa_lo = nullptr;  // attention output, [Kt_q]
  u32x4 *ha_hi = nullptr, *ha_lo = nullptr;  // SwiGLU output, [Kt_F]
  u32x4 *ua_hi = nullptr, *ua_lo = nullptr;  // fused rows u * g_fuse, [D, mt_max, Kt_H]
  int mt_max = 1;
  float* opart = nullptr;
  float2* ml = nullptr;
  float* pmax = nullptr;
  int* pidx = nullptr;
  u32x4* zero_tile = nullptr;
  Plan p_qkv, p_o, p_gu, p_down, p_lm, p_kvt;
  int attn_chunk = 128, attn_nchunks = 1;
  // debug capture
  bool debug = false;
  float *dbg_hidden = nullptr, *dbg_logits = nullptr, *dbg_fused = nullptr;
  int dbg_fused_n = 0;
  // captured draft blocks, keyed by the output buffer
  struct BlockGraph {
    int32_t* out;
    hipGraphExec_t exec;
  };
  std::vector<BlockGraph> graphs;
  bool use_graphs = true;
  // kernel timing
  int prof_kind = 0;
  std::vector<hipEvent_t> prof_ev;  // pairs
  int prof_n = 0;
  std::vector<void*> allocs;
  std::string err;
};

namespace {

int fail(dflare_handle* h, int code, const std::string& msg) {
  if (h) h->err = msg;
  else g_init_error = msg;
  return code;
}

#define HIP_OR_FAIL(h, call)                                                                     \
  do {                                                                                           \
    hipError_t e_ = (call);                                                                      \
    if (e_ != hipSuccess)                                                                        \
      return fail((h), DFLARE_ERR_HIP, std::string(#call ": ") + hipGetErrorString(e_));         \
  } while (0)

template <typename T>
int dev_alloc(dflare_handle* h, T** p, size_t bytes) {
  if (bytes == 0) bytes = 256;
  void* q = nullptr;
  hipError_t e = hipMalloc(&q, bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(h, DFLARE_ERR_OUT_OF_MEMORY, "hipMalloc of " + std::to_string(bytes) + " bytes failed");
  }
  h->allocs.push_back(q);
  *p = static_cast<T*>(q);
  return DFLARE_OK;
}

void drop_graphs(dflare_handle* h);

void free_all(dflare_handle* h) {
  drop_graphs(h);
  for (void* p : h->allocs) (void)hipFree(p);
  h->allocs.clear();
  for (hipEvent_t e : h->prof_ev) (void)hipEventDestroy(e);
  h->prof_ev.clear();
}

const int kProfMax = 8192;

// bracket one launch of kernel kind `k` with events when it is the profiled kind
void prof_mark(dflare_handle* h, int k, bool start) {
  if (h->prof_kind != k || h->prof_n >= kProfMax) return;
  const size_t ix = 2 * (size_t)h->prof_n + (start ? 0 : 1);
  while (h->prof_ev.size() <= ix) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) {
      h->prof_kind = 0;
      return;
    }
    h->prof_ev.push_back(e);
  }
  (void)hipEventRecord(h->prof_ev[ix], h->stream);
  if (!start) ++h->prof_n;
}

bool live(const dflare_handle* h) {
  std::lock_guard<std::mutex> lk(g_mu);
  return h && g_live.count(h) && h->magic == kMagic;
}

// Plan of a weight-streaming GEMM: output tiles per block and waves per block.  The defaults
// can be overridden with DFLARE_PLAN_<NAME>=nt,waves (used for tuning).
Plan make_plan(const char* name, int Nt, int nt, int waves) {
  char key[64];
  snprintf(key, sizeof key, "DFLARE_PLAN_%s", name);
  if (const char* env = getenv(key)) {
    int x = 0, y = 0;
    if (sscanf(env, "%d,%d", &x, &y) == 2 && gemm_shape_supported(x, y)) {
      nt = x;
      waves = y;
    }
  }
  Plan p;
  p.nt = nt;
  p.waves = waves;
  p.groups = ceil_div(Nt, nt);
  return p;
}

GemmArgs gemm_args(const dflare_handle* h, const u32x4* W, int Nt, int Kt) {
  GemmArgs a{};
  a.W = W;
  a.Nt = Nt;
  a.Kt = Kt;
  a.zero = h->zero_tile;
  a.eps = h->cfg.rms_eps;
  a.e.params = h->params;
  a.e.Lcap = h->Lcap;
  a.e.plane = h->cache_plane;
  a.e.hd = h->cfg.head_dim;
  a.e.rope = h->rope;
  a.e.B = h->cfg.block_size;
  return a;
}

int check_launch(dflare_handle* h, const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(h, DFLARE_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
  return DFLARE_OK;
}

int validate_config(const dflare_config* c) {
  if (!c) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "cfg is NULL");
  if (c->hidden <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0 || c->ffn <= 0 ||
      c->vocab <= 0 || c->n_draft_layers <= 0 || c->n_target_layers <= 0 || c->block_size <= 0 ||
      c->max_context <= 0 || c->max_new <= 0)
    return fail(nullptr, DFLARE_ERR_INVALID_ARG, "every size in dflare_config must be positive");
  if (!(c->rope_base > 0.f) || !(c->rms_eps >= 0.f) || !isfinite(c->rope_base) || !isfinite(c->rms_eps))
    return fail(nullptr, DFLARE_ERR_INVALID_ARG, "rope_base must be > 0 and rms_eps >= 0");
  if (c->n_q_heads % c->n_kv_heads)
    return fail(nullptr, DFLARE_ERR_INVALID_ARG, "n_q_heads must be a multiple of n_kv_heads");
  if (c->block_size > 16) return fail(nullptr, DFLARE_ERR_UNSUPPORTED, "block_size must be <= 16");
  if (c->head_dim != 64 && c->head_dim != 128) return fail(nullptr, DFLARE_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (c->hidden % 32 || c->ffn % 32 || (c->n_q_heads * c->head_dim) % 32)
    return fail(nullptr, DFLARE_ERR_UNSUPPORTED, "hidden, ffn and n_q_heads*head_dim must be multiples of 32");
  if ((c->n_q_heads / c->n_kv_heads) * c->block_size > 128)
    return fail(nullptr, DFLARE_ERR_UNSUPPORTED, "(n_q_heads / n_kv_heads) * block_size must be <= 128");
  if (c->n_target_layers > 64) return fail(nullptr, DFLARE_ERR_UNSUPPORTED, "n_target_layers must be <= 64");
  if (c->hidden > 8192) return fail(nullptr, DFLARE_ERR_UNSUPPORTED, "hidden must be <= 8192");
  if ((long)c->max_context + c->block_size > (1L << 30))
    return fail(nullptr, DFLARE_ERR_UNSUPPORTED, "max_context too large");
  return DFLARE_OK;
}

#define TRY(x)                         \
  do {                                 \
    int rc_ = (x);                     \
    if (rc_ != DFLARE_OK) return rc_;  \
  } while (0)

int build(dflare_handle* h, const dflare_weights* w) {
  const dflare_config& c = h->cfg;
  const int H = c.hidden, D = c.n_draft_layers, S = c.n_target_layers, F = c.ffn, V = c.vocab;
  const int hd = c.head_dim, B = c.block_size;
  h->q_dim = c.n_q_heads * hd;
  h->kv_dim = c.n_kv_heads * hd;
  const int q = h->q_dim, kv = h->kv_dim;
  h->Lcap = ceil_div((long)c.max_context + B, 64) * 64;
  h->Rpad = ceil_div((long)(c.n_q_heads / c.n_kv_heads) * B, 16) * 16;
  hipStream_t s = h->stream;

  // ---- plans
  const int Nt_qkv = (q + 2 * kv) / 16, Nt_o = H / 16, Nt_gu = 2 * F / 16, Nt_down = H / 16;
  const int Nt_lm = ceil_div(V, 16), Nt_kvt = 2 * kv / 16;
  const int Kt_H = H / 32, Kt_q = q / 32, Kt_F = F / 32;
  const int mt_max = ceil_div(c.max_new, 16);
  h->p_qkv = make_plan("QKV", Nt_qkv, 2, 16);
  h->p_o = make_plan("O", Nt_o, 1, 16);
  h->p_gu = make_plan("GU", Nt_gu, 4, 4);
  h->p_down = make_plan("DOWN", Nt_down, 1, 16);
  h->p_lm = make_plan("LM", Nt_lm, 4, 4);
  h->p_kvt = make_plan("KVT", Nt_kvt, 1, 16);
  if (const char* env = getenv("DFLARE_GRAPH")) h->use_graphs = atoi(env) != 0;
  if (const char* env = getenv("DFLARE_ATTN_CHUNK")) {
    int v = atoi(env);
    if (v == 64 || v == 128) h->attn_chunk = v;
  }
  // chunk c holds keys [c*chunk, (c+1)*chunk); the last one also the B block keys
  h->attn_nchunks = std::max(1, ceil_div((long)c.max_context, h->attn_chunk));

  // ---- packed weights
  h->s_qkv = (long)Nt_qkv * Kt_H * 64;
  h->s_o = (long)Nt_o * Kt_q * 64;
  h->s_gu = (long)Nt_gu * Kt_H * 64;
  h->s_down = (long)Nt_down * Kt_F * 64;
  h->s_kvt = (long)Nt_kvt * Kt_H * 64;
  TRY(dev_alloc(h, &h->w_qkv, (size_t)h->s_qkv * D * 16));
  TRY(dev_alloc(h, &h->w_o, (size_t)h->s_o * D * 16));
  TRY(dev_alloc(h, &h->w_gu, (size_t)h->s_gu * D * 16));
  TRY(dev_alloc(h, &h->w_down, (size_t)h->s_down * D * 16));
  TRY(dev_alloc(h, &h->w_kvt, (size_t)h->s_kvt * D * 16));
  TRY(dev_alloc(h, &h->w_lm, (size_t)Nt_lm * Kt_H * 64 * 16));
  TRY(dev_alloc(h, &h->embed, (size_t)V * H * 2));
  const uint16_t* wq = (const uint16_t*)w->wq;
  const uint16_t* wkd = (const uint16_t*)w->wk_d;
  const uint16_t* wvd = (const uint16_t*)w->wv_d;
  const uint16_t* wkt = (const uint16_t*)w->wk_t;
  const uint16_t* wvt = (const uint16_t*)w->wv_t;
  const uint16_t* wo = (const uint16_t*)w->wo;
  const uint16_t* wg = (const uint16_t*)w->w_gate;
  const uint16_t* wu = (const uint16_t*)w->w_up;
  const uint16_t* wd = (const uint16_t*)w->w_down;
  for (int i = 0; i < D; ++i) {
    u32x4* dq = h->w_qkv + i * h->s_qkv;
    launch_pack(s, dq, wq + (long)i * q * H, nullptr, q, H, 0, q / 16, Kt_H, PACK_ROPE, hd);
    launch_pack(s, dq, wkd + (long)i * kv * H, nullptr, kv, H, q / 16, kv / 16, Kt_H, PACK_ROPE, hd);
    launch_pack(s, dq, wvd + (long)i * kv * H, nullptr, kv, H, (q + kv) / 16, kv / 16, Kt_H, PACK_IDENTITY, hd);
    u32x4* dk = h->w_kvt + i * h->s_kvt;
    launch_pack(s, dk, wkt + (long)i * kv * H, nullptr, kv, H, 0, kv / 16, Kt_H, PACK_ROPE, hd);
    launch_pack(s, dk, wvt + (long)i * kv * H, nullptr, kv, H, kv / 16, kv / 16, Kt_H, PACK_IDENTITY, hd);
    launch_pack(s, h->w_o + i * h->s_o, wo + (long)i * H * q, nullptr, H, q, 0, Nt_o, Kt_q, PACK_IDENTITY, hd);
    launch_pack(s, h->w_gu + i * h->s_gu, wg + (long)i * F * H, wu + (long)i * F * H, F, H, 0, Nt_gu, Kt_H,
                PACK_SWIGLU, hd);
    launch_pack(s, h->w_down + i * h->s_down, wd + (long)i * H * F, nullptr, H, F, 0, Nt_down, Kt_F,
                PACK_IDENTITY, hd);
  }
  launch_pack(s, h->w_lm, (const uint16_t*)w->lm_head, nullptr, V, H, 0, Nt_lm, Kt_H, PACK_IDENTITY, hd);
  TRY(check_launch(h, "weight packing"));
  HIP_OR_FAIL(h, hipMemcpyAsync(h->embed, w->embed, (size_t)V * H * 2, hipMemcpyDeviceToDevice, s));

  // ---- gains (fp32), alpha
  TRY(dev_alloc(h, &h->g_fuse, (size_t)D * H * 4));
  TRY(dev_alloc(h, &h->g_attn, (size_t)D * H * 4));
  TRY(dev_alloc(h, &h->g_mlp, (size_t)D * H * 4));
  TRY(dev_alloc(h, &h->g_final, (size_t)H * 4));
  launch_bf16_to_f32(s, h->g_fuse, (const uint16_t*)w->fuse_norm, (long)D * H);
  launch_bf16_to_f32(s, h->g_attn, (const uint16_t*)w->attn_norm, (long)D * H);
  launch_bf16_to_f32(s, h->g_mlp, (const uint16_t*)w->mlp_norm, (long)D * H);
  launch_bf16_to_f32(s, h->g_final, (const uint16_t*)w->final_norm, (long)H);
  TRY(check_launch(h, "gain conversion"));
  TRY(dev_alloc(h, &h->alpha, (size_t)D * S * 4));
  HIP_OR_FAIL(h, hipMemcpyAsync(h->alpha, h->alpha_host.data(), (size_t)D * S * 4, hipMemcpyHostToDevice, s));

  // ---- context cache, rotary table
  // per layer: K (or V^T) as two bf16 planes, hi then lo (value ~= hi + lo)
  h->cache_plane = (long)c.n_kv_heads * h->Lcap * hd;
  h->cache_layer_stride = 2 * h->cache_plane;
  TRY(dev_alloc(h, &h->kc, (size_t)h->cache_layer_stride * D * 2));
  TRY(dev_alloc(h, &h->vt, (size_t)h->cache_layer_stride * D * 2));
  HIP_OR_FAIL(h, hipMemsetAsync(h->kc, 0, (size_t)h->cache_layer_stride * D * 2, s));
  HIP_OR_FAIL(h, hipMemsetAsync(h->vt, 0, (size_t)h->cache_layer_stride * D * 2, s));
  {
    const int half = hd / 2;
    std::vector<float2> tab((size_t)h->Lcap * half);
    for (int p = 0; p < h->Lcap; ++p)
      for (int m = 0; m < half; ++m) {
        const double th = (double)p * pow((double)c.rope_base, -2.0 * m / hd);
        tab[(size_t)p * half + m] = make_float2((float)cos(th), (float)sin(th));
      }
    TRY(dev_alloc(h, &h->rope, tab.size() * sizeof(float2)));
    HIP_OR_FAIL(h, hipMemcpy(h->rope, tab.data(), tab.size() * sizeof(float2), hipMemcpyHostToDevice));
  }

  // ---- step scratch
  TRY(dev_alloc(h, &h->params, sizeof(StepParams)));
  TRY(dev_alloc(h, &h->zero_tile, 64 * 16));
  HIP_OR_FAIL(h, hipMemsetAsync(h->zero_tile, 0, 64 * 16, s));
  TRY(dev_alloc(h, &h->ids, 64 * 4));
  TRY(dev_alloc(h, &h->X, (size_t)16 * H * 4));
  TRY(dev_alloc(h, &h->Xstats, (size_t)16 * (H / 16) * 4));
  TRY(dev_alloc(h, &h->Q, (size_t)16 * q * 4));
  TRY(dev_alloc(h, &h->Ustats, (size_t)D * c.max_new * (H / 16) * 4));
  h->mt_max = mt_max;
  {
    const size_t pad = 64;
    const size_t nx = (size_t)Kt_H + pad, no = (size_t)Kt_q + pad, nh = (size_t)Kt_F + pad;
    const size_t nu = (size_t)D * mt_max * Kt_H + pad;
    u32x4** bufs[8] = {&h->xa_hi, &h->xa_lo, &h->oa_hi, &h->oa_lo, &h->ha_hi, &h->ha_lo, &h->ua_hi, &h->ua_lo};
    const size_t tiles[8] = {nx, nx, no, no, nh, nh, nu, nu};
    for (int b = 0; b < 8; ++b) {
      TRY(dev_alloc(h, bufs[b], tiles[b] * 1024));
      HIP_OR_FAIL(h, hipMemsetAsync(*bufs[b], 0, tiles[b] * 1024, s));
    }
  }
  TRY(dev_alloc(h, &h->opart, (size_t)h->attn_nchunks * c.n_kv_heads * h->Rpad * hd * 4));
  TRY(dev_alloc(h, &h->ml, (size_t)h->attn_nchunks * c.n_kv_heads * h->Rpad * sizeof(float2)));
  TRY(dev_alloc(h, &h->pmax, (size_t)16 * h->p_lm.groups * 4));
  TRY(dev_alloc(h, &h->pidx, (size_t)16 * h->p_lm.groups * 4));
  HIP_OR_FAIL(h, hipStreamSynchronize(s));
  return DFLARE_OK;
}

// Every kernel of a draft block after the prologue.  The launch sequence and its arguments
// depend only on the handle and `out`, so it can be captured once in a HIP graph and replayed.
int enqueue_block_body(dflare_handle* h, int32_t* out) {
  const dflare_config& c = h->cfg;
  const int H = c.hidden, D = c.n_draft_layers, F = c.ffn, B = c.block_size, hd = c.head_dim;
  const int q = h->q_dim, kv = h->kv_dim;
  hipStream_t s = h->stream;
  launch_embed(s, h->embed, h->ids, c.vocab, H, B, h->X, h->Xstats, h->g_attn, h->xa_hi, h->xa_lo);

  AttnArgs at{};
  at.params = h->params;
  at.Q = h->Q;
  at.B = B;
  at.n_q = c.n_q_heads;
  at.n_kv = c.n_kv_heads;
  at.q_dim = q;
  at.Lcap = h->Lcap;
  at.plane = h->cache_plane;
  at.Rpad = h->Rpad;
  at.qscale = (float)(1.4426950408889634 / sqrt((double)hd));
  at.opart = h->opart;
  at.ml = h->ml;
  at.oa_hi = h->oa_hi;
  at.oa_lo = h->oa_lo;
  at.oa_Kt = q / 32;

  for (int i = 0; i < D; ++i) {
    uint16_t* kc = h->kc + i * h->cache_layer_stride;
    uint16_t* vt = h->vt + i * h->cache_layer_stride;
    {  // RMSNorm + Q / K^d / V^d + RoPE, block K/V into cache slots L..L+B-1
      GemmArgs a = gemm_args(h, h->w_qkv + i * h->s_qkv, (q + 2 * kv) / 16, H / 32);
      a.Ahi = h->xa_hi; a.Alo = h->xa_lo; a.M = B;
      a.stats = h->Xstats; a.n_stat = H / 16; a.inv_dim = 1.0f / H;
      a.e.out = h->Q; a.e.ldo = q; a.e.kc = kc; a.e.vt = vt;
      a.e.q_tiles = q / 16; a.e.kv_tiles = kv / 16;
      prof_mark(h, DFLARE_K_QKV, true);
      launch_gemm(s, EPI_QKV, h->p_qkv.nt, h->p_qkv.waves, a, 1, 1);
      prof_mark(h, DFLARE_K_QKV, false);
    }
    at.kc = kc;
    at.vt = vt;
    prof_mark(h, DFLARE_K_ATTN, true);
    launch_attention(s, at, hd, h->attn_chunk, h->attn_nchunks);
    launch_attn_combine(s, at, hd, h->attn_chunk, h->attn_nchunks);
    prof_mark(h, DFLARE_K_ATTN, false);
    {  // X += O W_O^T
      GemmArgs a = gemm_args(h, h->w_o + i * h->s_o, H / 16, q / 32);
      a.Ahi = h->oa_hi; a.Alo = h->oa_lo; a.M = B;
      a.e.out = h->X; a.e.ldo = H; a.e.stats_out = h->Xstats; a.e.n_stat_out = H / 16;
      a.e.na_hi = (uint32_t*)h->xa_hi; a.e.na_lo = (uint32_t*)h->xa_lo; a.e.na_Kt = H / 32;
      a.e.next_gain = h->g_mlp + (long)i * H;
      prof_mark(h, DFLARE_K_O, true);
      launch_gemm(s, EPI_RESID, h->p_o.nt, h->p_o.waves, a, 1, 1);
      prof_mark(h, DFLARE_K_O, false);
    }
    {  // RMSNorm + gate/up + SwiGLU
      GemmArgs a = gemm_args(h, h->w_gu + i * h->s_gu, 2 * F / 16, H / 32);
      a.Ahi = h->xa_hi; a.Alo = h->xa_lo; a.M = B;
      a.stats = h->Xstats; a.n_stat = H / 16; a.inv_dim = 1.0f / H;
      a.e.na_hi = (uint32_t*)h->ha_hi; a.e.na_lo = (uint32_t*)h->ha_lo; a.e.na_Kt = F / 32;
      prof_mark(h, DFLARE_K_GATE_UP, true);
      launch_gemm(s, EPI_SWIGLU, h->p_gu.nt, h->p_gu.waves, a, 1, 1);
      prof_mark(h, DFLARE_K_GATE_UP, false);
    }
    {  // X += H W_down^T
      GemmArgs a = gemm_args(h, h->w_down + i * h->s_down, H / 16, F / 32);
      a.Ahi = h->ha_hi; a.Alo = h->ha_lo; a.M = B;
      a.e.out = h->X; a.e.ldo = H; a.e.stats_out = h->Xstats; a.e.n_stat_out = H / 16;
      a.e.na_hi = (uint32_t*)h->xa_hi; a.e.na_lo = (uint32_t*)h->xa_lo; a.e.na_Kt = H / 32;
      a.e.next_gain = (i + 1 < D) ? h->g_attn + (long)(i + 1) * H : h->g_final;
      prof_mark(h, DFLARE_K_DOWN, true);
      launch_gemm(s, EPI_RESID, h->p_down.nt, h->p_down.waves, a, 1, 1);
      prof_mark(h, DFLARE_K_DOWN, false);
    }
    if (h->debug)
      HIP_OR_FAIL(h, hipMemcpyAsync(h->dbg_hidden + (long)i * B * H, h->X, (size_t)B * H * 4,
                                    hipMemcpyDeviceToDevice, s));
  }
  {  // final RMSNorm + LM head + argmax
    GemmArgs a = gemm_args(h, h->w_lm, ceil_div(c.vocab, 16), H / 32);
    a.Ahi = h->xa_hi; a.Alo = h->xa_lo; a.M = B;
    a.stats = h->Xstats; a.n_stat = H / 16; a.inv_dim = 1.0f / H;
    a.e.vocab = c.vocab; a.e.pmax = h->pmax; a.e.pidx = h->pidx;
    a.e.logits = h->debug ? h->dbg_logits : nullptr;
    prof_mark(h, DFLARE_K_LM_HEAD, true);
    launch_gemm(s, EPI_ARGMAX, h->p_lm.nt, h->p_lm.waves, a, 1, 1);
    launch_argmax_combine(s, h->pmax, h->pidx, h->p_lm.groups, B, out);
    prof_mark(h, DFLARE_K_LM_HEAD, false);
  }
  return check_launch(h, "draft_block");
}

void drop_graphs(dflare_handle* h) {
  for (auto& g : h->graphs) (void)hipGraphExecDestroy(g.exec);
  h->graphs.clear();
}

int run_draft_block(dflare_handle* h, const int32_t* ids, const int32_t* positions_host, int32_t* out) {
  const int B = h->cfg.block_size;
  hipStream_t s = h->stream;
  StepParams sp{};
  sp.L = h->L;
  sp.n_new = 0;
  for (int b = 0; b < B; ++b) sp.pos[b] = positions_host ? positions_host[b] : h->L + b;
  launch_prologue(s, h->params, sp, ids, h->ids, B);
  // Graph replay needs a capturable (non-null) stream; debug capture and kernel timing
  // insert extra work between the kernels, so they run eagerly.
  const bool graph = h->use_graphs && s != nullptr && !h->debug && h->prof_kind == 0;
  if (!graph) return enqueue_block_body(h, out);
  for (auto& g : h->graphs)
    if (g.out == out) {
      HIP_OR_FAIL(h, hipGraphLaunch(g.exec, s));
      return DFLARE_OK;
    }
  hipGraph_t graph_def = nullptr;
  HIP_OR_FAIL(h, hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal));
  const int rc = enqueue_block_body(h, out);
  const hipError_t ce = hipStreamEndCapture(s, &graph_def);
  if (rc != DFLARE_OK) {
    if (graph_def) (void)hipGraphDestroy(graph_def);
    return rc;
  }
  if (ce != hipSuccess) return fail(h, DFLARE_ERR_HIP, std::string("graph capture: ") + hipGetErrorString(ce));
  hipGraphExec_t exec = nullptr;
  const hipError_t ie = hipGraphInstantiate(&exec, graph_def, nullptr, nullptr, 0);
  (void)hipGraphDestroy(graph_def);
  if (ie != hipSuccess) return fail(h, DFLARE_ERR_HIP, std::string("graph instantiate: ") + hipGetErrorString(ie));
  if (h->graphs.size() >= 4) {  // keep the four most recent output buffers
    (void)hipGraphExecDestroy(h->graphs.front().exec);
    h->graphs.erase(h->graphs.begin());
  }
  h->graphs.push_back({out, exec});
  HIP_OR_FAIL(h, hipGraphLaunch(exec, s));
  return DFLARE_OK;
}

}  // namespace

extern "C" {

int dflare_init(const dflare_config* cfg, const dflare_weights* w, const float* fusion_logits, void* stream,
                dflare_handle** out) {
  g_init_error.clear();
  if (!out) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  TRY(validate_config(cfg));
  if (!w || !w->embed || !w->lm_head || !w->wq || !w->wk_d || !w->wv_d || !w->wk_t || !w->wv_t || !w->wo ||
      !w->w_gate || !w->w_up || !w->w_down)
    return fail(nullptr, DFLARE_ERR_INVALID_ARG, "a required weight pointer is NULL");
  if (!fusion_logits) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "fusion_logits is NULL");
  const int D = cfg->n_draft_layers, S = cfg->n_target_layers;
  // alpha^(i) = softmax(W^fuse_{i,:}) in double precision, cached as float (Sec. 4.1)
  std::vector<float> alpha((size_t)D * S);
  for (int i = 0; i < D; ++i) {
    const float* row = fusion_logits + (size_t)i * S;
    double mx = -INFINITY;
    for (int j = 0; j < S; ++j) {
      if (isnan(row[j]) || (isinf(row[j]) && row[j] > 0))
        return fail(nullptr, DFLARE_ERR_INVALID_ARG, "fusion logits contain NaN or +inf");
      mx = std::max(mx, (double)row[j]);
    }
    if (!isfinite(mx)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "a fusion-logit row has no finite entry");
    double z = 0.0;
    for (int j = 0; j < S; ++j) z += exp((double)row[j] - mx);
    for (int j = 0; j < S; ++j) alpha[(size_t)i * S + j] = (float)(exp((double)row[j] - mx) / z);
  }
  dflare_handle* h = new dflare_handle();
  h->cfg = *cfg;
  h->stream = (hipStream_t)stream;
  h->alpha_host = alpha;
  int rc = build(h, w);
  if (rc != DFLARE_OK) {
    g_init_error = h->err;
    (void)hipStreamSynchronize(h->stream);
    free_all(h);
    delete h;
    return rc;
  }
  {
    std::lock_guard<std::mutex> lk(g_mu);
    g_live.insert(h);
  }
  *out = h;
  return DFLARE_OK;
}

int dflare_fuse_append(dflare_handle* h, const void* target_hidden, int32_t n_new) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  if (!target_hidden) return fail(h, DFLARE_ERR_INVALID_ARG, "target_hidden is NULL");
  if (n_new < 1 || n_new > h->cfg.max_new)
    return fail(h, DFLARE_ERR_INVALID_ARG, "n_new must be in [1, max_new]");
  if ((long)h->L + n_new > h->cfg.max_context)
    return fail(h, DFLARE_ERR_CONTEXT_FULL, "append would exceed max_context");
  const dflare_config& c = h->cfg;
  const int H = c.hidden, D = c.n_draft_layers, S = c.n_target_layers;
  hipStream_t s = h->stream;
  prof_mark(h, DFLARE_K_FUSE, true);
  launch_fuse(s, (const uint16_t*)target_hidden, n_new, S, H, D, h->alpha, h->g_fuse, h->Ustats, h->ua_hi,
              h->ua_lo, c.max_new, h->mt_max, h->params, h->L);
  prof_mark(h, DFLARE_K_FUSE, false);
  GemmArgs a = gemm_args(h, h->w_kvt, 2 * h->kv_dim / 16, H / 32);
  a.w_layer_stride = h->s_kvt;
  a.Ahi = h->ua_hi; a.Alo = h->ua_lo; a.a_layer_stride = (long)h->mt_max * (H / 32) * 64;
  a.stats = h->Ustats; a.stats_layer_stride = (long)c.max_new * (H / 16); a.n_stat = H / 16;
  a.inv_dim = 1.0f / H;
  a.e.kc = h->kc; a.e.vt = h->vt; a.e.cache_layer_stride = h->cache_layer_stride;
  a.e.q_tiles = 0; a.e.kv_tiles = h->kv_dim / 16;
  prof_mark(h, DFLARE_K_KV_T, true);
  launch_gemm(s, EPI_KVT, h->p_kvt.nt, h->p_kvt.waves, a, D, ceil_div(n_new, 16));
  prof_mark(h, DFLARE_K_KV_T, false);
  if (h->debug) {
    launch_fused_rows(s, h->ua_hi, h->ua_lo, h->Ustats, n_new, H, D, c.max_new, h->mt_max, c.rms_eps,
                      h->dbg_fused);
    h->dbg_fused_n = n_new;
  }
  int rc = check_launch(h, "fuse_append");
  if (rc != DFLARE_OK) return rc;
  h->L += n_new;
  return DFLARE_OK;
}

int dflare_draft_block(dflare_handle* h, const int32_t* block_ids, int32_t* draft_tokens) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  if (!block_ids || !draft_tokens) return fail(h, DFLARE_ERR_INVALID_ARG, "block_ids / draft_tokens is NULL");
  return run_draft_block(h, block_ids, nullptr, draft_tokens);
}

int dflare_draft_block_pos(dflare_handle* h, const int32_t* block_ids, const int32_t* positions,
                           int32_t* draft_tokens) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  if (!block_ids || !draft_tokens || !positions)
    return fail(h, DFLARE_ERR_INVALID_ARG, "block_ids / positions / draft_tokens is NULL");
  for (int b = 0; b < h->cfg.block_size; ++b)
    if (positions[b] < 0 || positions[b] >= h->Lcap)
      return fail(h, DFLARE_ERR_INVALID_ARG, "a position is outside [0, max_context + block_size)");
  return run_draft_block(h, block_ids, positions, draft_tokens);
}

int dflare_truncate(dflare_handle* h, int32_t new_len) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  if (new_len < 0 || new_len > h->L) return fail(h, DFLARE_ERR_INVALID_ARG, "new_len must be in [0, L]");
  h->L = new_len;
  return DFLARE_OK;
}

int dflare_context_len(const dflare_handle* h, int32_t* out) {
  if (!live(h) || !out) return DFLARE_ERR_INVALID_ARG;
  *out = h->L;
  return DFLARE_OK;
}

int dflare_set_stream(dflare_handle* h, void* stream) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  h->stream = (hipStream_t)stream;
  return DFLARE_OK;
}

int dflare_destroy(dflare_handle* h) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  {
    std::lock_guard<std::mutex> lk(g_mu);
    g_live.erase(h);
  }
  (void)hipStreamSynchronize(h->stream);
  free_all(h);
  h->magic = 0;
  delete h;
  return DFLARE_OK;
}

const char* dflare_status_str(int status) {
  switch (status) {
    case DFLARE_OK: return "ok";
    case DFLARE_ERR_INVALID_ARG: return "invalid argument";
    case DFLARE_ERR_OUT_OF_MEMORY: return "out of device memory";
    case DFLARE_ERR_CONTEXT_FULL: return "context full";
    case DFLARE_ERR_HIP: return "HIP runtime error";
    case DFLARE_ERR_UNSUPPORTED: return "unsupported shape";
    default: return "unknown status";
  }
}

const char* dflare_last_error(const dflare_handle* h) {
  if (!h) return g_init_error.c_str();
  if (!live(h)) return "invalid handle";
  return h->err.c_str();
}

int dflare_debug_capture(dflare_handle* h, int on) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  const dflare_config& c = h->cfg;
  if (on && !h->dbg_hidden) {
    TRY(dev_alloc(h, &h->dbg_hidden, (size_t)c.n_draft_layers * c.block_size * c.hidden * 4));
    TRY(dev_alloc(h, &h->dbg_logits, (size_t)c.block_size * c.vocab * 4));
    TRY(dev_alloc(h, &h->dbg_fused, (size_t)c.n_draft_layers * c.max_new * c.hidden * 4));
  }
  h->debug = on != 0;
  return DFLARE_OK;
}

int dflare_debug_read(dflare_handle* h, int what, int layer, float* host_out, int64_t count) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  if (!host_out) return fail(h, DFLARE_ERR_INVALID_ARG, "host_out is NULL");
  const dflare_config& c = h->cfg;
  const int H = c.hidden, B = c.block_size, hd = c.head_dim, nkv = c.n_kv_heads;
  const bool needs_layer = what == DFLARE_DBG_FUSED || what == DFLARE_DBG_KCACHE || what == DFLARE_DBG_VCACHE ||
                           what == DFLARE_DBG_HIDDEN;
  if (needs_layer && (layer < 0 || layer >= c.n_draft_layers))
    return fail(h, DFLARE_ERR_INVALID_ARG, "layer out of range");
  if (what != DFLARE_DBG_ALPHA && what != DFLARE_DBG_KCACHE && what != DFLARE_DBG_VCACHE && !h->dbg_hidden)
    return fail(h, DFLARE_ERR_INVALID_ARG, "debug capture was never enabled");
  HIP_OR_FAIL(h, hipStreamSynchronize(h->stream));
  switch (what) {
    case DFLARE_DBG_ALPHA: {
      const int64_t n = (int64_t)c.n_draft_layers * c.n_target_layers;
      if (count < n) return fail(h, DFLARE_ERR_INVALID_ARG, "host buffer too small");
      HIP_OR_FAIL(h, hipMemcpy(host_out, h->alpha, n * 4, hipMemcpyDeviceToHost));
      return DFLARE_OK;
    }
    case DFLARE_DBG_FUSED: {
      const int64_t n = (int64_t)h->dbg_fused_n * H;
      if (count < n) return fail(h, DFLARE_ERR_INVALID_ARG, "host buffer too small");
      HIP_OR_FAIL(h, hipMemcpy(host_out, h->dbg_fused + (long)layer * h->dbg_fused_n * H, n * 4,
                               hipMemcpyDeviceToHost));
      return DFLARE_OK;
    }
    case DFLARE_DBG_HIDDEN: {
      const int64_t n = (int64_t)B * H;
      if (count < n) return fail(h, DFLARE_ERR_INVALID_ARG, "host buffer too small");
      HIP_OR_FAIL(h, hipMemcpy(host_out, h->dbg_hidden + (long)layer * B * H, n * 4, hipMemcpyDeviceToHost));
      return DFLARE_OK;
    }
    case DFLARE_DBG_LOGITS: {
      const int64_t n = (int64_t)B * c.vocab;
      if (count < n) return fail(h, DFLARE_ERR_INVALID_ARG, "host buffer too small");
      HIP_OR_FAIL(h, hipMemcpy(host_out, h->dbg_logits, n * 4, hipMemcpyDeviceToHost));
      return DFLARE_OK;
    }
    case DFLARE_DBG_KCACHE:
    case DFLARE_DBG_VCACHE: {
      const int64_t n = (int64_t)h->L * nkv * hd;
      if (count < n) return fail(h, DFLARE_ERR_INVALID_ARG, "host buffer too small");
      std::vector<uint16_t> raw((size_t)h->cache_layer_stride);
      const uint16_t* src = (what == DFLARE_DBG_KCACHE ? h->kc : h->vt) + (long)layer * h->cache_layer_stride;
      HIP_OR_FAIL(h, hipMemcpy(raw.data(), src, raw.size() * 2, hipMemcpyDeviceToHost));
      for (int p = 0; p < h->L; ++p)
        for (int g = 0; g < nkv; ++g)
          for (int d = 0; d < hd; ++d) {
            const size_t ix = (what == DFLARE_DBG_KCACHE) ? ((size_t)g * h->Lcap + p) * hd + d
                                                          : ((size_t)g * hd + d) * h->Lcap + p;
            const uint32_t hb = (uint32_t)raw[ix] << 16, lb = (uint32_t)raw[ix + h->cache_plane] << 16;
            float fh, fl;
            memcpy(&fh, &hb, 4);
            memcpy(&fl, &lb, 4);
            host_out[((size_t)p * nkv + g) * hd + d] = fh + fl;
          }
      return DFLARE_OK;
    }
    default: return fail(h, DFLARE_ERR_INVALID_ARG, "unknown debug tensor");
  }
}

int dflare_profile_begin(dflare_handle* h, int kind) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  if (kind < 0 || kind > DFLARE_K_KV_T) return fail(h, DFLARE_ERR_INVALID_ARG, "unknown kernel kind");
  h->prof_kind = kind;
  h->prof_n = 0;
  return DFLARE_OK;
}

int dflare_profile_end(dflare_handle* h, double* total_ms, int32_t* launches) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  if (!total_ms || !launches) return fail(h, DFLARE_ERR_INVALID_ARG, "NULL output");
  HIP_OR_FAIL(h, hipStreamSynchronize(h->stream));
  double t = 0.0;
  for (int i = 0; i < h->prof_n; ++i) {
    float ms = 0.f;
    HIP_OR_FAIL(h, hipEventElapsedTime(&ms, h->prof_ev[2 * i], h->prof_ev[2 * i + 1]));
    t += ms;
  }
  *total_ms = t;
  *launches = h->prof_n;
  h->prof_kind = 0;
  h->prof_n = 0;
  return DFLARE_OK;
}

int dflare_kernel_stats(const dflare_handle* h, int32_t* out, int32_t count) {
  if (!live(h) || !out) return DFLARE_ERR_INVALID_ARG;
  const int32_t v[2] = {2 + 6 * h->cfg.n_draft_layers + 2, 2};
  for (int i = 0; i < count && i < 2; ++i) out[i] = v[i];
  return DFLARE_OK;
}

}  // extern "C"
