// Host runtime and C ABI of the DFlare draft step (see include/dflare.h).
//
// One handle owns: the re-packed weights, the cached fusion weights alpha, the
// per-draft-layer context cache of every sequence slot (K as [n_kv, Lcap, hd], V
// transposed as [n_kv, hd, Lcap], fp16), a rotary table, and the activation buffers of
// one draft block and of one batched draft step.  fuse_append enqueues two kernels (fusion,
// context K/V projection); draft_block enqueues one persistent kernel (or, on request,
// the same kernel once per phase).  Values that change between calls (L,
// n_new, positions, the block ids pointer) travel as kernel arguments.
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <unordered_set>
#include <utility>
#include <vector>

#include <hip/hip_ext.h>

#include "batched.h"
#include "dflare.h"
#include "dflare_impl.h"

using namespace dflare;

namespace {

const uint32_t kMagic = 0xDF1A2E00u;

std::mutex g_mu;
std::unordered_set<const dflare_handle*> g_live;
thread_local std::string g_init_error;

int ceil_div(long a, long b) { return (int)((a + b - 1) / b); }

// IEEE binary16 bits -> float (exact)
float half_to_float(uint16_t hbits) {
  const uint32_t sign = (uint32_t)(hbits >> 15) << 31, e = (hbits >> 10) & 31u, m = hbits & 1023u;
  float v;
  if (e == 0) v = ldexpf((float)m, -24);                        // zero, subnormal
  else if (e == 31) v = m ? NAN : INFINITY;
  else v = ldexpf((float)(m | 1024u), (int)e - 25);
  uint32_t u;
  memcpy(&u, &v, 4);
  u |= sign;
  memcpy(&v, &u, 4);
  return v;
}

}  // namespace

namespace {
struct GemmPlan {  // chunk width and K split of one GEMM phase kind
  int tn = 8, kg = 1;
};
}  // namespace

struct dflare_handle {
  uint32_t magic = kMagic;
  dflare_config cfg{};
  hipStream_t stream = nullptr;
  int device = 0;
  std::vector<int> Ls;  // context length of each sequence slot (slot 0: the batch-1 calls)
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
  float2* rope = nullptr;
  u32x4* zero_tile = nullptr;
  // fuse_append scratch
  float* Ustats = nullptr;
  u32x4 *ua_hi = nullptr, *ua_lo = nullptr;  // fused rows u * g_fuse, [D, mt_max, Kt_H]
  int mt_max = 1;
  int kvt_nt = 2, kvt_waves = 8;
  // draft block
  int blocks = 0;          // work-groups of the draft kernel
  int phases = 0;
  bool persistent = true;
  bool coop_ok = false;    // the device keeps one work-group per CU resident
  bool coop_launch = false;  // DFLARE_OPT_COOPERATIVE: the persistent kernel through the cooperative launch
  int draft_sig = 0;         // signature of the GEMM plans (draft_plan_sig) when a kernel is built for them
  bool generic_draft = false;  // DFLARE_OPT_GENERIC_KERNEL: the generic draft kernel whatever the plans
  GemmPlan plan[PH_COUNT];
  int attn_nch = 1;
  int attn_chunk = 128;
  float* X = nullptr;
  float* XS = nullptr;
  long xs_stride = 0;
  u32x4* XA = nullptr;
  long xa_stride = 0;
  float* Q = nullptr;
  long q_stride = 0;
  uint16_t* OP = nullptr;  // draft-block attention partials (fp16)
  float2* ML = nullptr;
  u32x4* OA = nullptr;
  long oa_stride = 0;
  u32x4* HA = nullptr;
  long ha_stride = 0;
  float* pmax = nullptr;
  int* pidx = nullptr;
  float* part = nullptr;
  DraftArgs* args_dev = nullptr;  // device copy of the draft kernel's fixed arguments
  unsigned* sync = nullptr;  // barrier counters, the LM-head completion counter, split-K counters
  unsigned bar_epoch = 0, done_epoch = 0;
  unsigned acnt_epoch = 0;  // value of every attention arrival counter (grows by D * chunks per draft block)
  unsigned qcnt_epoch = 0;  // value of every Q/K/V tile counter (grows by D * (G + 2) * hd / 16 per draft block)
  int* err_host = nullptr;   // host-mapped barrier time-out flag
  int* err_dev = nullptr;
  // Context length of slot 0 kept on the device (after dflare_accept_async): two words used
  // in turn, Ldev[lcur] the current one, so that a verification step reads the length the
  // draft step used while it writes the next one; L_hi bounds it from above.  kdev: k when
  // the caller passes no word for it.
  int32_t* Ldev = nullptr;
  int32_t* kdev = nullptr;
  bool dev_len = false;
  int lcur = 0;
  long L_hi = 0;
  bool trace = false;
  bool capture_persistent = false;  // debug capture written by the persistent launch itself
  unsigned long long* trace_buf = nullptr;
  // debug capture
  bool debug = false;
  float *dbg_hidden = nullptr, *dbg_logits = nullptr, *dbg_fused = nullptr;
  int dbg_fused_n = 0;
  // kernel timing
  int prof_kind = 0;
  std::vector<hipEvent_t> prof_ev;  // pairs
  int prof_n = 0;
  // candidate selection: temperature 0 greedy, else Gumbel-max draws (draw counts draft calls)
  float temperature = 0.f;
  unsigned long long seed = 0;
  unsigned draw = 0;
  // batched draft step
  int cus = 0;
  long seq_stride = 0;     // cache elements of one sequence slot (all layers)
  int b_mt = 1;            // m-tiles of the largest batched call
  float *bX = nullptr, *bQ = nullptr, *bOP = nullptr;
  float2* bML = nullptr;
  u32x4 *bA = nullptr, *bOA = nullptr, *bHA = nullptr;  // fp16 A fragments of the GEMM inputs
  u32x4* bU = nullptr;     // fp16 A fragments of the fused rows of a batched append, per layer
  // variants: K/V bias of the folded +FC layer [D][2 kv]; DFlash FC weights (bf16 tiles and
  // their fp16 copy), bias, and the fragments of its input rows and of the context rows
  float* kv_bias = nullptr;
  u32x4 *w_fc = nullptr, *h_fc = nullptr;
  float* fc_bias = nullptr;
  u32x4 *bCat = nullptr, *bC = nullptr;
  // fp16 copies of the packed weight tiles, made on first use of the batched path
  u32x4 *h_qkv = nullptr, *h_o = nullptr, *h_gu = nullptr, *h_down = nullptr, *h_kvt = nullptr, *h_lm = nullptr;
  float* bpart = nullptr;  // split-K partial tiles
  long bpart_floats = 0;
  unsigned* bcnt = nullptr;
  float* bpmax = nullptr;
  int* bpidx = nullptr;
  float* dbg_blogits = nullptr;
  int dbg_blogits_rows = 0;
  std::vector<void*> allocs;
  std::vector<std::pair<void*, size_t>> uc_blocks;  // uncached counter blocks (returned to the pool)
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

#define TRY(x)                         \
  do {                                 \
    int rc_ = (x);                     \
    if (rc_ != DFLARE_OK) return rc_;  \
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

// zero-filled device allocation
template <typename T>
int dev_zalloc(dflare_handle* h, T** p, size_t bytes) {
  TRY(dev_alloc(h, p, bytes));
  HIP_OR_FAIL(h, hipMemsetAsync(*p, 0, bytes, h->stream));
  return DFLARE_OK;
}

// Uncached device memory for the arrival counters that work-groups poll (grid barriers,
// attention and LM-head counts): a poll of uncached memory returns sooner while the CU
// streams weights (about 1 us per barrier under load; 10 us per Qwen3-8B-shaped draft
// block).  A block that a kernel has read is never handed back to the driver (freeing
// uncached memory has been followed by wrong contents in later allocations on this
// platform): released blocks stay in a per-device pool for the next handle until the process
// ends.
std::mutex g_uc_mu;
std::vector<std::pair<int, std::pair<void*, size_t>>> g_uc_pool;  // (device, (block, bytes))

template <typename T>
int uc_zalloc(dflare_handle* h, T** p, size_t bytes) {
  void* q = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_uc_mu);
    for (size_t i = 0; i < g_uc_pool.size(); ++i)
      if (g_uc_pool[i].first == h->device && g_uc_pool[i].second.second == bytes) {
        q = g_uc_pool[i].second.first;
        g_uc_pool.erase(g_uc_pool.begin() + (long)i);
        break;
      }
  }
  if (!q) {
    hipError_t e = hipExtMallocWithFlags(&q, bytes, hipDeviceMallocUncached);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return fail(h, DFLARE_ERR_OUT_OF_MEMORY, "uncached allocation of " + std::to_string(bytes) + " bytes failed");
    }
  }
  h->uc_blocks.push_back({q, bytes});
  *p = static_cast<T*>(q);
  HIP_OR_FAIL(h, hipMemsetAsync(q, 0, bytes, h->stream));
  return DFLARE_OK;
}

void free_all(dflare_handle* h) {
  for (void* p : h->allocs) (void)hipFree(p);
  h->allocs.clear();
  {
    std::lock_guard<std::mutex> lk(g_uc_mu);
    for (const auto& b : h->uc_blocks) g_uc_pool.push_back({h->device, b});
  }
  h->uc_blocks.clear();
  if (h->err_host) (void)hipHostFree(h->err_host);
  h->err_host = nullptr;
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
  if (c->block_size > kMaxBlock) return fail(nullptr, DFLARE_ERR_UNSUPPORTED, "block_size must be <= 16");
  if (c->head_dim != 64 && c->head_dim != 128) return fail(nullptr, DFLARE_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (c->hidden % 32 || c->ffn % 32 || (c->n_q_heads * c->head_dim) % 32)
    return fail(nullptr, DFLARE_ERR_UNSUPPORTED, "hidden, ffn and n_q_heads*head_dim must be multiples of 32");
  if ((c->n_q_heads / c->n_kv_heads) * c->block_size > 128)
    return fail(nullptr, DFLARE_ERR_UNSUPPORTED, "(n_q_heads / n_kv_heads) * block_size must be <= 128");
  if (c->n_q_heads / c->n_kv_heads > 8 || c->n_kv_heads > kMaxKvHeads)
    return fail(nullptr, DFLARE_ERR_UNSUPPORTED, "n_q_heads / n_kv_heads must be <= 8 and n_kv_heads <= 128");
  if (c->n_target_layers > 64) return fail(nullptr, DFLARE_ERR_UNSUPPORTED, "n_target_layers must be <= 64");
  if (c->hidden > 8192) return fail(nullptr, DFLARE_ERR_UNSUPPORTED, "hidden must be <= 8192");
  if ((long)c->max_context + c->block_size > (1L << 30))
    return fail(nullptr, DFLARE_ERR_UNSUPPORTED, "max_context too large");
  if (c->max_batch < 0 || c->max_batch > kMaxSeq)
    return fail(nullptr, DFLARE_ERR_UNSUPPORTED, "max_batch must be in [0, 64]");
  if (c->variant & ~15) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "unknown variant flags");
  if ((c->variant & DFLARE_VARIANT_DFLASH) && (c->variant & ~DFLARE_VARIANT_DFLASH))
    return fail(nullptr, DFLARE_ERR_INVALID_ARG, "DFLASH does not combine with other variant flags");
  return DFLARE_OK;
}

// GEMM plan of a phase kind (see DraftArgs::tn / kg).  Candidates: kg in {1, 2, 4, 8}
// dividing the work-group count (kg > 1 only where the epilogue is linear in the sum and
// a range fits one chunk of <= 8 tiles), tn the smallest of 2, 3, 4, 5, 6, 8 that holds a range
// (8 when a range needs several chunks).  Cost, in KiB streamed by the busiest work-group:
// its weight tiles, plus a quarter of its A-fragment and padding re-reads (L2 hits), plus
// for a split the partial tiles the last work-group reads back and a fixed 16 for the
// extra round trip.  DFLARE_PLAN_<NAME>=tn,kg overrides the choice (tuning, tests).
bool plan_ok(int tn, int kg, int Nt, int blocks, bool allow_split) {
  if (tn < 2 || tn > 8 || tn == 7) return false;
  if (kg < 1 || kg > kMaxSplit || (kg & (kg - 1)) || blocks % kg) return false;
  if (kg > 1 && (!allow_split || ceil_div(Nt, blocks / kg) > tn)) return false;
  return true;
}

// only_tn != 0 restricts the candidates to that chunk width (none may fit: cost 1e300);
// *cost_out receives the chosen plan's cost.
GemmPlan choose_plan(const char* name, int Nt, int Kt, int blocks, bool allow_split, int only_tn = 0,
                     double* cost_out = nullptr) {
  GemmPlan best;
  double best_cost = 1e300;
  for (int kg = 1; kg <= kMaxSplit; kg *= 2) {
    if (blocks % kg || (kg > 1 && !allow_split)) continue;
    const int T = ceil_div(Nt, blocks / kg);
    if (kg > 1 && T > kTNMax) continue;
    int tn = kTNMax;
    for (int c : {2, 3, 4, 5, 6, 8})
      if (c >= T) {
        tn = c;
        break;
      }
    if (only_tn && tn != only_tn) continue;
    const int nch = ceil_div(T, tn);
    const int kpart = ceil_div(Kt, kg);
    const double cost = (double)T * kpart + 0.25 * ((double)nch * 2 * kpart + (double)(nch * tn - T) * kpart) +
                        (kg > 1 ? 16.0 + 2.0 * (kg - 1) * T : 0.0);
    if (cost < best_cost - 1e-9) {
      best_cost = cost;
      best.tn = tn;
      best.kg = kg;
    }
  }
  if (cost_out) *cost_out = best_cost;
  char key[64];
  snprintf(key, sizeof key, "DFLARE_PLAN_%s", name);
  if (const char* env = getenv(key)) {
    int tn = 0, kg = 0;
    if (sscanf(env, "%d,%d", &tn, &kg) == 2 && plan_ok(tn, kg, Nt, blocks, allow_split)) {
      best.tn = tn;
      best.kg = kg;
    }
  }
  return best;
}

// The output and down projections run the same epilogue: with one chunk width they share one
// GEMM body in the draft kernel, so a layer runs from less code (each phase's epilogue runs
// once per layer and is fetched anew when the layer's code does not stay in the instruction
// cache).  Their plans take the common width with the lowest summed cost when that sum is
// within 5% of the two independent choices' (at the Qwen3-4B shape the down projection's
// 6 x 8 -> 4 x 4 raised the summed cost 3% and made the draft block 680 -> 671 us).  Not
// applied when either plan is set by the environment.
void share_resid_width(GemmPlan& po, GemmPlan& pd, int Nt_o, int Kt_o, int Nt_d, int Kt_d, int blocks) {
  if (getenv("DFLARE_PLAN_O") || getenv("DFLARE_PLAN_DOWN")) return;
  double co = 0, cd = 0;
  choose_plan("O", Nt_o, Kt_o, blocks, true, 0, &co);
  choose_plan("DOWN", Nt_d, Kt_d, blocks, true, 0, &cd);
  if (po.tn == pd.tn) return;
  double best = 1e300;
  GemmPlan bo = po, bd = pd;
  for (int tn : {2, 3, 4, 5, 6, 8}) {
    double xo = 0, xd = 0;
    const GemmPlan qo = choose_plan("O", Nt_o, Kt_o, blocks, true, tn, &xo);
    const GemmPlan qd = choose_plan("DOWN", Nt_d, Kt_d, blocks, true, tn, &xd);
    if (xo + xd < best) {
      best = xo + xd;
      bo = qo;
      bd = qd;
    }
  }
  if (best <= 1.05 * (co + cd)) {
    po = bo;
    pd = bd;
  }
}

// K split of a batched GEMM (1 where the epilogue needs whole sums before it can start
// or the tiles outnumber the arrival counters): the deepest split whose work-groups still
// fit one per CU (tiles x kg <= CUs), each part keeping at least 8 k-tiles.  A sweep of the
// split at the Qwen3-8B shape with 512 rows picked exactly these (Q/K/V 2, output 4, down 4,
// gate/up 1, the 8-layer context K/V of a ~270-row append 1); an earlier cost fit in k-tiles
// per work-group chose 3 for Q/K/V, 23% slower.
// DFLARE_BSPLIT_<NAME>=kg overrides the choice (tuning).
int bgemm_split(int cus, const char* name, int Nt, int Mt, int Kt, int layers, bool allow, int nw = kBNW) {
  const long tiles = (long)bgemm_groups(Nt, Mt, nw) * layers;
  if (!allow || tiles > kBCounters) return 1;
  int best = 1;
  for (int kg : {2, 3, 4, 6, 8})
    if (tiles * kg <= cus && Kt >= 8 * kg) best = kg;
  char key[64];
  snprintf(key, sizeof key, "DFLARE_BSPLIT_%s", name);
  if (const char* env = getenv(key)) {
    const int v = atoi(env);
    if (v >= 1 && v <= kBSplitMax && v <= Kt) best = v;
  }
  return best;
}

// Output-tile width of a batched GEMM (n-tiles per wave, 4 or 3): 3 where its work-groups
// (with their K split) fill whole rounds of two per CU better, e.g. gate/up at 512 rows
// (384 work-groups of 4 leave half the CUs with one, 512 of 3 give every CU two) and Q/K/V
// (192 vs 256 work-groups on 256 CUs).  The LM head keeps 4 (its partial maxima are laid
// out per 256 columns).  DFLARE_BNW_<NAME>=3|4 overrides the choice (tuning).
int bgemm_nw(int cus, const char* name, int Nt, int Mt, int Kt, int layers, bool allow) {
  auto fill = [&](int nw) {
    const long wgs = (long)bgemm_groups(Nt, Mt, nw) * layers * bgemm_split(cus, name, Nt, Mt, Kt, layers, allow, nw);
    const long slots = 2L * cus;
    return (double)wgs / (double)(((wgs + slots - 1) / slots) * slots);
  };
  int nw = allow && fill(3) > fill(kBNW) + 1e-9 ? 3 : kBNW;
  char key[64];
  snprintf(key, sizeof key, "DFLARE_BNW_%s", name);
  if (const char* env = getenv(key)) {
    const int v = atoi(env);
    if (allow && (v == 3 || v == kBNW)) nw = v;
  }
  return nw;
}

DraftArgs draft_args(const dflare_handle* h);
int ensure_f16_weights(dflare_handle* h);

int build(dflare_handle* h, const dflare_weights* w) {
  const dflare_config& c = h->cfg;
  const int H = c.hidden, D = c.n_draft_layers, S = c.n_target_layers, F = c.ffn, V = c.vocab;
  const int hd = c.head_dim, B = c.block_size;
  h->q_dim = c.n_q_heads * hd;
  h->kv_dim = c.n_kv_heads * hd;
  const int q = h->q_dim, kv = h->kv_dim;
  // 8 spare slots: a 16-byte V^T piece that starts at the last block key stays inside a row
  h->Lcap = ceil_div((long)c.max_context + B + 8, 64) * 64;
  h->Rpad = ceil_div((long)(c.n_q_heads / c.n_kv_heads) * B, 16) * 16;
  hipStream_t s = h->stream;
  HIP_OR_FAIL(h, hipGetDevice(&h->device));

  const int Nt_qkv = (q + 2 * kv) / 16, Nt_o = H / 16, Nt_gu = 2 * F / 16, Nt_down = H / 16;
  const int Nt_lm = ceil_div(V, 16), Nt_kvt = 2 * kv / 16;
  const int Kt_H = H / 32, Kt_q = q / 32, Kt_F = F / 32;
  const int mt_max = ceil_div(c.max_new, 16);

  // ---- launch shape of the draft block: one work-group of kThreads per CU
  int cus = 0;
  HIP_OR_FAIL(h, hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, h->device));
  h->cus = cus;
  int coop = 0;
  HIP_OR_FAIL(h, hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, h->device));
  const int per_cu = draft_blocks_per_cu(hd, 0);
  h->coop_ok = coop != 0 && per_cu >= 1;
  h->blocks = cus;
  if (const char* env = getenv("DFLARE_BLOCKS")) {
    const int v = atoi(env);
    if (v >= 16 && v <= cus) h->blocks = v;
  }
  if (h->blocks > kMaxBlocks) h->blocks = kMaxBlocks;
  h->persistent = h->coop_ok;
  if (const char* env = getenv("DFLARE_PERSISTENT"))
    if (atoi(env) == 0) h->persistent = false;
  h->phases = phase_count(D);
  h->plan[PH_QKV] = choose_plan("QKV", Nt_qkv, Kt_H, h->blocks, true);
  h->plan[PH_O] = choose_plan("O", Nt_o, Kt_q, h->blocks, true);
  h->plan[PH_GU] = choose_plan("GU", Nt_gu, Kt_H, h->blocks, true);
  h->plan[PH_DOWN] = choose_plan("DOWN", Nt_down, Kt_F, h->blocks, true);
  h->plan[PH_LM] = choose_plan("LM", Nt_lm, Kt_H, h->blocks, false);
  share_resid_width(h->plan[PH_O], h->plan[PH_DOWN], Nt_o, Kt_q, Nt_down, Kt_F, h->blocks);
  {
    const int sig = draft_plan_sig(h->plan[PH_QKV].tn, h->plan[PH_O].tn, h->plan[PH_GU].tn, h->plan[PH_DOWN].tn);
    if (draft_specialized(hd, sig) && draft_blocks_per_cu(hd, sig) >= 1) h->draft_sig = sig;
  }
  if (getenv("DFLARE_VERBOSE"))
    fprintf(stderr, "dflare: %d work-groups; GEMM plans (tn,kg) qkv %d,%d o %d,%d gate/up %d,%d down %d,%d lm %d,%d\n",
            h->blocks, h->plan[PH_QKV].tn, h->plan[PH_QKV].kg, h->plan[PH_O].tn, h->plan[PH_O].kg,
            h->plan[PH_GU].tn, h->plan[PH_GU].kg, h->plan[PH_DOWN].tn, h->plan[PH_DOWN].kg, h->plan[PH_LM].tn,
            h->plan[PH_LM].kg);
  if (const char* env = getenv("DFLARE_PLAN_KVT")) {
    int x = 0, y = 0;
    if (sscanf(env, "%d,%d", &x, &y) == 2 && kvt_shape_supported(x, y)) {
      h->kvt_nt = x;
      h->kvt_waves = y;
    }
  }
  // attention chunks of the draft block: 128 context keys per chunk at head size 128, 256 at 64
  h->attn_chunk = hd == 64 ? 256 : 128;
  h->attn_nch = std::max(1, ceil_div((long)c.max_context, h->attn_chunk));

  // ---- packed weights
  h->s_qkv = (long)Nt_qkv * Kt_H * 64;
  h->s_o = (long)Nt_o * Kt_q * 64;
  h->s_gu = (long)Nt_gu * Kt_H * 64;
  h->s_down = (long)Nt_down * Kt_F * 64;
  h->s_kvt = (long)Nt_kvt * Kt_H * 64;
  TRY(dev_zalloc(h, &h->w_qkv, (size_t)h->s_qkv * D * 16 + kWeightSpare));
  TRY(dev_zalloc(h, &h->w_o, (size_t)h->s_o * D * 16 + kWeightSpare));
  TRY(dev_zalloc(h, &h->w_gu, (size_t)h->s_gu * D * 16 + kWeightSpare));
  TRY(dev_zalloc(h, &h->w_down, (size_t)h->s_down * D * 16 + kWeightSpare));
  TRY(dev_alloc(h, &h->w_kvt, (size_t)h->s_kvt * D * 16));
  TRY(dev_zalloc(h, &h->w_lm, (size_t)Nt_lm * Kt_H * 64 * 16 + kWeightSpare));
  TRY(dev_alloc(h, &h->embed, (size_t)V * H * 2));
  const uint16_t* wq = (const uint16_t*)w->wq;
  const uint16_t* wkd = (const uint16_t*)w->wk_d;
  const uint16_t* wvd = (const uint16_t*)w->wv_d;
  // context projections: W^t (Eq. 4), or the draft layer's own W^d (-KVProj, DFlash)
  const bool shared_kv = c.variant & (DFLARE_VARIANT_SHARED_KV | DFLARE_VARIANT_DFLASH);
  const uint16_t* wkt = (const uint16_t*)(shared_kv ? w->wk_d : w->wk_t);
  const uint16_t* wvt = (const uint16_t*)(shared_kv ? w->wv_d : w->wv_t);
  // +FC: W' = W W_pfc per layer (double precision, rounded to bf16), b' = W b_pfc in fp32
  uint16_t *fold_k = nullptr, *fold_v = nullptr;
  if (c.variant & DFLARE_VARIANT_POST_FC) {
    TRY(dev_alloc(h, &fold_k, (size_t)kv * H * 2));
    TRY(dev_alloc(h, &fold_v, (size_t)kv * H * 2));
    TRY(dev_alloc(h, &h->kv_bias, (size_t)D * 2 * kv * 4));
  }
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
    const uint16_t* src_k = wkt + (long)i * kv * H;
    const uint16_t* src_v = wvt + (long)i * kv * H;
    if (c.variant & DFLARE_VARIANT_POST_FC) {
      const uint16_t* pfc = (const uint16_t*)w->post_fc + (long)i * H * H;
      const uint16_t* pb = w->post_fc_bias ? (const uint16_t*)w->post_fc_bias + (long)i * H : nullptr;
      launch_compose(s, fold_k, src_k, pfc, kv, H, H);
      launch_compose(s, fold_v, src_v, pfc, kv, H, H);
      launch_matvec(s, h->kv_bias + (long)i * 2 * kv, src_k, pb, kv, H);
      launch_matvec(s, h->kv_bias + (long)i * 2 * kv + kv, src_v, pb, kv, H);
      src_k = fold_k;
      src_v = fold_v;
    }
    launch_pack(s, dk, src_k, nullptr, kv, H, 0, kv / 16, Kt_H, PACK_ROPE, hd);
    launch_pack(s, dk, src_v, nullptr, kv, H, kv / 16, kv / 16, Kt_H, PACK_IDENTITY, hd);
    launch_pack(s, h->w_o + i * h->s_o, wo + (long)i * H * q, nullptr, H, q, 0, Nt_o, Kt_q, PACK_IDENTITY, hd);
    launch_pack(s, h->w_gu + i * h->s_gu, wg + (long)i * F * H, wu + (long)i * F * H, F, H, 0, Nt_gu, Kt_H,
                PACK_SWIGLU, hd);
    launch_pack(s, h->w_down + i * h->s_down, wd + (long)i * H * F, nullptr, H, F, 0, Nt_down, Kt_F,
                PACK_IDENTITY, hd);
  }
  launch_pack(s, h->w_lm, (const uint16_t*)w->lm_head, nullptr, V, H, 0, Nt_lm, Kt_H, PACK_IDENTITY, hd);
  if (c.variant & DFLARE_VARIANT_DFLASH) {  // W_fc [H, S*H] as tiles of H/16 outputs x S*H/32 k
    TRY(dev_alloc(h, &h->w_fc, (size_t)(H / 16) * (S * H / 32) * 64 * 16));
    launch_pack(s, h->w_fc, (const uint16_t*)w->fc, nullptr, H, S * H, 0, H / 16, S * H / 32, PACK_IDENTITY, hd);
    TRY(dev_zalloc(h, &h->fc_bias, (size_t)H * 4));
    if (w->fc_bias) launch_bf16_to_f32(s, h->fc_bias, (const uint16_t*)w->fc_bias, (long)H);
  }
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
  // per layer: K (or V^T) in fp16
  h->cache_layer_stride = (long)c.n_kv_heads * h->Lcap * hd;
  h->seq_stride = h->cache_layer_stride * D;
  h->Ls.assign(c.max_batch, 0);
  TRY(dev_zalloc(h, &h->kc, (size_t)h->seq_stride * c.max_batch * 2));
  TRY(dev_zalloc(h, &h->vt, (size_t)h->seq_stride * c.max_batch * 2));
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
  TRY(dev_zalloc(h, &h->zero_tile, 64 * 16));

  // ---- fuse_append scratch
  h->mt_max = mt_max;
  TRY(dev_zalloc(h, &h->Ustats, (size_t)D * c.max_new * (H / 16) * 4));
  TRY(dev_zalloc(h, &h->ua_hi, (size_t)D * mt_max * Kt_H * 1024));
  TRY(dev_zalloc(h, &h->ua_lo, (size_t)D * mt_max * Kt_H * 1024));

  // ---- draft-block activations.  Rows >= B of every A-fragment and stats buffer stay zero.
  const int stages = 2 * D + 1;
  TRY(dev_zalloc(h, &h->X, (size_t)kMaxBlock * H * 4));
  h->xs_stride = (long)(H / 16) * kStatsPad;
  TRY(dev_zalloc(h, &h->XS, (size_t)stages * h->xs_stride * 4));
  h->xa_stride = 2L * (Kt_H + kKtPad) * 64;
  TRY(dev_zalloc(h, &h->XA, (size_t)stages * h->xa_stride * 16));
  h->q_stride = (long)kMaxBlock * q;
  TRY(dev_zalloc(h, &h->Q, (size_t)D * h->q_stride * 4));
  {  // per layer and chunk: G * 16 rows for every KV head
    const size_t rows = (size_t)D * h->attn_nch * c.n_q_heads * 16;
    TRY(dev_zalloc(h, &h->OP, rows * hd * 2));
    TRY(dev_zalloc(h, &h->ML, rows * sizeof(float2)));
  }
  h->oa_stride = 2L * (Kt_q + kKtPad) * 64;
  TRY(dev_zalloc(h, &h->OA, (size_t)D * h->oa_stride * 16));
  h->ha_stride = 2L * (Kt_F + kKtPad) * 64;
  TRY(dev_zalloc(h, &h->HA, (size_t)D * h->ha_stride * 16));
  TRY(dev_zalloc(h, &h->pmax, (size_t)h->blocks * kStatsPad * 4));
  TRY(dev_zalloc(h, &h->pidx, (size_t)h->blocks * kStatsPad * 4));
  // split-K partial tiles: one area per GEMM phase kind (tagged per use, see gemm_phase)
  TRY(dev_zalloc(h, &h->part, (size_t)kSplitKinds * h->blocks * kTNMax * 1024));
  TRY(uc_zalloc(h, &h->sync, kSyncBytes));
  TRY(dev_zalloc(h, &h->Ldev, 4 * sizeof(int32_t)));
  h->kdev = h->Ldev + 2;

  // ---- batched draft step: activations of max_batch * B rows
  {
    h->b_mt = ceil_div((long)c.max_batch * B, 16);
    const long rows = (long)h->b_mt * 16;
    TRY(dev_zalloc(h, &h->bX, (size_t)rows * H * 4));
    TRY(dev_zalloc(h, &h->bQ, (size_t)rows * q * 4));
    TRY(dev_zalloc(h, &h->bA, (size_t)h->b_mt * Kt_H * 1024));
    TRY(dev_zalloc(h, &h->bOA, (size_t)h->b_mt * Kt_q * 1024));
    TRY(dev_zalloc(h, &h->bHA, (size_t)h->b_mt * Kt_F * 1024));
    TRY(dev_zalloc(h, &h->bU, (size_t)D * mt_max * Kt_H * 1024));
    if (c.variant & DFLARE_VARIANT_DFLASH) {
      TRY(dev_zalloc(h, &h->bCat, (size_t)mt_max * (S * H / 32) * 1024));
      TRY(dev_zalloc(h, &h->bC, (size_t)mt_max * Kt_H * 1024));
    }
    // partial tiles of the largest split of any call shape
    long part = 0;
    auto need = [&](const char* name, int Nt, int mt, int Kt, int layers) {
      for (int nw : {kBNW, 3}) {  // either tile width (the per-tile partial scales with it)
        const int kg = bgemm_split(h->cus, name, Nt, mt, Kt, layers, true, nw);
        if (kg > 1) part = std::max(part, (long)bgemm_groups(Nt, mt, nw) * layers * kg * kBPartFloats);
      }
    };
    for (int mt = 1; mt <= h->b_mt; ++mt) {
      need("QKV", Nt_qkv, mt, Kt_H, 1);
      need("O", Nt_o, mt, Kt_q, 1);
      need("GU", Nt_gu, mt, Kt_H, 1);
      need("DOWN", Nt_down, mt, Kt_F, 1);
    }
    for (int mt = 1; mt <= mt_max; ++mt) {
      need("KVT", Nt_kvt, mt, Kt_H, D);
      if (c.variant & DFLARE_VARIANT_DFLASH) need("FC", H / 16, mt, S * H / 32, 1);
    }
    h->bpart_floats = part;
    TRY(dev_alloc(h, &h->bpart, (size_t)std::max(part, 64L) * 4));
    TRY(dev_zalloc(h, &h->bcnt, (size_t)kBCounters * 128));
    const long items = (long)c.max_batch * ceil_div((long)c.max_context + B, kBKeys) * c.n_kv_heads;
    TRY(dev_alloc(h, &h->bOP, (size_t)items * h->Rpad * hd * 4));
    TRY(dev_alloc(h, &h->bML, (size_t)items * h->Rpad * sizeof(float2)));
    const long ng_lm = ceil_div(Nt_lm, kBN);
    TRY(dev_alloc(h, &h->bpmax, (size_t)ng_lm * rows * 4));
    TRY(dev_alloc(h, &h->bpidx, (size_t)ng_lm * rows * 4));
  }
  if (c.max_batch > 1 || (c.variant & DFLARE_VARIANT_DFLASH)) TRY(ensure_f16_weights(h));
  HIP_OR_FAIL(h, hipHostMalloc((void**)&h->err_host, 64, hipHostMallocMapped | hipHostMallocCoherent));
  *(volatile int*)h->err_host = 0;
  HIP_OR_FAIL(h, hipHostGetDevicePointer((void**)&h->err_dev, h->err_host, 0));
  {
    const DraftArgs a = draft_args(h);
    TRY(dev_alloc(h, &h->args_dev, sizeof(DraftArgs)));
    HIP_OR_FAIL(h, hipMemcpy(h->args_dev, &a, sizeof(DraftArgs), hipMemcpyHostToDevice));
  }
  HIP_OR_FAIL(h, hipStreamSynchronize(s));
  return DFLARE_OK;
}

DraftArgs draft_args(const dflare_handle* h) {
  const dflare_config& c = h->cfg;
  DraftArgs a{};
  a.H = c.hidden;
  a.F = c.ffn;
  a.V = c.vocab;
  a.D = c.n_draft_layers;
  a.B = c.block_size;
  a.hd = c.head_dim;
  a.n_q = c.n_q_heads;
  a.n_kv = c.n_kv_heads;
  a.Lcap = h->Lcap;
  a.Rpad = h->Rpad;
  a.chunk = h->attn_chunk;
  a.nch = h->attn_nch;
  a.eps = c.rms_eps;
  a.qscale = (float)(1.4426950408889634 / sqrt((double)c.head_dim));
  const int H = c.hidden, Kt_H = H / 32, q = c.n_q_heads * c.head_dim, kv = c.n_kv_heads * c.head_dim;
  for (int k = 0; k < PH_COUNT; ++k) {
    a.tn[k] = h->plan[k].tn;
    a.kg[k] = h->plan[k].kg;
    int Nt = 0, Kt = 0;
    switch (k) {
      case PH_QKV: Nt = (q + 2 * kv) / 16; Kt = Kt_H; break;
      case PH_O: Nt = H / 16; Kt = q / 32; break;
      case PH_GU: Nt = 2 * c.ffn / 16; Kt = Kt_H; break;
      case PH_DOWN: Nt = H / 16; Kt = c.ffn / 32; break;
      case PH_LM: Nt = (c.vocab + 15) / 16; Kt = Kt_H; break;
      default: break;
    }
    const int R = h->blocks / std::max(a.kg[k], 1);
    a.nq[k] = Nt / R;
    a.nr[k] = Nt % R;
    a.kq[k] = Kt / std::max(a.kg[k], 1);
    a.kr[k] = Kt % std::max(a.kg[k], 1);
  }
  a.embed = h->embed;
  a.w_qkv = h->w_qkv;
  a.w_o = h->w_o;
  a.w_gu = h->w_gu;
  a.w_down = h->w_down;
  a.w_lm = h->w_lm;
  a.s_qkv = h->s_qkv;
  a.s_o = h->s_o;
  a.s_gu = h->s_gu;
  a.s_down = h->s_down;
  a.g_attn = h->g_attn;
  a.g_mlp = h->g_mlp;
  a.g_final = h->g_final;
  a.zero = h->zero_tile;
  a.rope = h->rope;
  a.kc = h->kc;
  a.vt = h->vt;
  a.cache_layer = h->cache_layer_stride;
  a.X = h->X;
  a.XS = h->XS;
  a.xs_stride = h->xs_stride;
  a.XA = h->XA;
  a.xa_stride = h->xa_stride;
  a.Q = h->Q;
  a.q_stride = h->q_stride;
  a.OP = h->OP;
  a.ML = h->ML;
  a.OA = h->OA;
  a.oa_stride = h->oa_stride;
  a.HA = h->HA;
  a.ha_stride = h->ha_stride;
  a.pmax = h->pmax;
  a.pidx = h->pidx;
  a.bar = h->sync;
  a.done = h->sync + kBarCounters * 32;
  a.part = h->part;
  a.kcnt = h->sync + 1024;
  a.acnt = h->sync + kAttnCntOff / 4;
  a.qcnt = h->sync + kQkvCntOff / 4;
  a.err = h->err_dev;
  return a;
}

DraftCall draft_call(const dflare_handle* h, const int32_t* ids, const int32_t* positions_host, int32_t* out) {
  const dflare_config& c = h->cfg;
  DraftCall d{};
  // with the length on the device (never together with host positions) the kernel adds it
  d.L = h->dev_len ? 0 : h->Ls[0];
  d.Lp = h->dev_len ? h->Ldev + h->lcur : nullptr;
  for (int b = 0; b < kMaxBlock; ++b) d.pos[b] = (b < c.block_size) ? (positions_host ? positions_host[b] : d.L + b) : 0;
  d.ids = ids;
  d.tokens = out;
  d.logits = h->debug ? h->dbg_logits : nullptr;
  d.hidden = (h->debug && h->capture_persistent && h->persistent) ? h->dbg_hidden : nullptr;
  d.bar_epoch = h->bar_epoch;
  d.done_epoch = h->done_epoch;
  d.acnt_base = h->acnt_epoch;
  d.qcnt_base = h->qcnt_epoch;
  d.trace = h->trace ? h->trace_buf : nullptr;
  d.inv_temp = h->temperature > 0.f ? 1.0f / h->temperature : 0.f;
  d.draw = h->draw;
  d.seed = h->seed;
  return d;
}

int prof_kind_of(int phase_kind) {
  switch (phase_kind) {
    case PH_QKV: return DFLARE_K_QKV;
    case PH_ATTN:
    case PH_COMB: return DFLARE_K_ATTN;
    case PH_O: return DFLARE_K_O;
    case PH_GU: return DFLARE_K_GATE_UP;
    case PH_DOWN: return DFLARE_K_DOWN;
    case PH_LM: return DFLARE_K_LM_HEAD;
    default: return 0;
  }
}

int run_draft_block(dflare_handle* h, const int32_t* ids, const int32_t* positions_host, int32_t* out) {
  const dflare_config& c = h->cfg;
  hipStream_t s = h->stream;
  if (*(volatile int*)h->err_host) {  // an earlier persistent launch timed out at a grid barrier
    HIP_OR_FAIL(h, hipStreamSynchronize(s));
    HIP_OR_FAIL(h, hipMemsetAsync(h->sync, 0, kSyncBytes, s));
    HIP_OR_FAIL(h, hipMemsetAsync(h->part, 0, (size_t)kSplitKinds * h->blocks * kTNMax * 1024, s));
    HIP_OR_FAIL(h, hipStreamSynchronize(s));
    h->bar_epoch = h->done_epoch = h->acnt_epoch = h->qcnt_epoch = 0;
    *(volatile int*)h->err_host = 0;
    h->persistent = false;
    return fail(h, DFLARE_ERR_HIP,
                "a grid barrier of an earlier draft_block timed out; its tokens are invalid and the handle "
                "now runs one launch per phase");
  }
  const int P = h->phases;
  // counters are monotonic across launches; start again from zero long before they wrap
  // (split-K counters reach (done_epoch + 1) * D * kg <= (done_epoch + 1) * D * 8)
  // (every layer adds the chunk capacity to each attention counter, whatever the length)
  // (every layer's Q/K/V phase adds each KV head's tile count, (G + 2) * hd / 16, to its counter)
  const unsigned attn_adds = (unsigned)c.n_draft_layers * (unsigned)h->attn_nch;
  const unsigned qkv_adds =
      (unsigned)c.n_draft_layers * (unsigned)(c.n_q_heads / c.n_kv_heads + 2) * (unsigned)(c.head_dim / 16);
  if (h->bar_epoch + (unsigned)P > (1u << 24) || h->done_epoch + 1u > (1u << 22) ||
      ((uint64_t)h->done_epoch + 1u) * (uint64_t)c.n_draft_layers * kMaxSplit >= (1ull << 31) ||
      (uint64_t)h->acnt_epoch + attn_adds >= (1ull << 31) || (uint64_t)h->qcnt_epoch + qkv_adds >= (1ull << 31)) {
    // the split-K partial tags follow done_epoch: start them again from cleared areas
    HIP_OR_FAIL(h, hipMemsetAsync(h->sync, 0, kSyncBytes, s));
    HIP_OR_FAIL(h, hipMemsetAsync(h->part, 0, (size_t)kSplitKinds * h->blocks * kTNMax * 1024, s));
    h->bar_epoch = h->done_epoch = h->acnt_epoch = h->qcnt_epoch = 0;
  }
  if (h->trace && !h->trace_buf) TRY(dev_zalloc(h, &h->trace_buf, (size_t)h->blocks * kTraceSlots * P * 8));
  if (h->trace) HIP_OR_FAIL(h, hipMemsetAsync(h->trace_buf, 0, (size_t)h->blocks * kTraceSlots * P * 8, s));
  const DraftCall dc = draft_call(h, ids, positions_host, out);
  const int hd = c.head_dim, sig = h->generic_draft ? 0 : h->draft_sig;
  const bool split = !h->persistent || (h->debug && !h->capture_persistent) ||
                     (h->prof_kind >= DFLARE_K_QKV && h->prof_kind <= DFLARE_K_LM_HEAD);
  prof_mark(h, DFLARE_K_DRAFT, true);
  if (!split) {
    HIP_OR_FAIL(h, launch_draft(s, h->args_dev, dc, hd, sig, h->blocks, 0, P, h->coop_launch));
    // a grid barrier before every phase but the first and the attention and combine phases
    h->bar_epoch += (unsigned)(P - 1 - 2 * c.n_draft_layers);
  } else {
    for (int p = 0; p < P; ++p) {
      int kind, layer;
      phase_of(p, c.n_draft_layers, kind, layer);
      const int pk = prof_kind_of(kind);
      const bool open = pk && (kind != PH_COMB);  // attention + combine are timed together
      if (open) prof_mark(h, pk, true);
      HIP_OR_FAIL(h, launch_draft(s, h->args_dev, dc, hd, sig, h->blocks, p, p + 1, false));
      if (pk && kind != PH_ATTN) prof_mark(h, pk, false);
      if (h->debug && kind == PH_DOWN)
        HIP_OR_FAIL(h, hipMemcpyAsync(h->dbg_hidden + (long)layer * c.block_size * c.hidden, h->X,
                                      (size_t)c.block_size * c.hidden * 4, hipMemcpyDeviceToDevice, s));
    }
  }
  h->done_epoch += 1;
  h->acnt_epoch += attn_adds;  // every attention item of every layer counted once
  h->qcnt_epoch += qkv_adds;   // every Q/K/V tile of every layer counted once
  if (h->temperature > 0.f) ++h->draw;
  prof_mark(h, DFLARE_K_DRAFT, false);
  return check_launch(h, "draft_block");
}

// Bring a device-resident length of slot 0 back to the host (waits for the stream).
int settle_len(dflare_handle* h) {
  if (!h->dev_len) return DFLARE_OK;
  HIP_OR_FAIL(h, hipStreamSynchronize(h->stream));
  int32_t L = 0;
  HIP_OR_FAIL(h, hipMemcpy(&L, h->Ldev + h->lcur, sizeof(L), hipMemcpyDeviceToHost));
  if (L < 0 || L > h->L_hi) return fail(h, DFLARE_ERR_HIP, "device-resident context length out of range");
  h->Ls[0] = L;
  h->dev_len = false;
  return DFLARE_OK;
}

// n_seq distinct slots in range
int check_seqs(dflare_handle* h, int32_t n_seq, const int32_t* seq) {
  TRY(settle_len(h));
  if (n_seq < 1 || n_seq > h->cfg.max_batch) return fail(h, DFLARE_ERR_INVALID_ARG, "n_seq must be in [1, max_batch]");
  if (!seq) return fail(h, DFLARE_ERR_INVALID_ARG, "seq is NULL");
  std::vector<char> seen(h->cfg.max_batch, 0);
  for (int i = 0; i < n_seq; ++i) {
    if (seq[i] < 0 || seq[i] >= h->cfg.max_batch)
      return fail(h, DFLARE_ERR_INVALID_ARG, "a sequence slot is outside [0, max_batch)");
    if (seen[seq[i]]) return fail(h, DFLARE_ERR_INVALID_ARG, "sequence slots must be distinct");
    seen[seq[i]] = 1;
  }
  return DFLARE_OK;
}

// fp16 copies of the packed weights for the batched GEMMs (allocated and converted once)
int ensure_f16_weights(dflare_handle* h) {
  if (h->h_lm) return DFLARE_OK;
  const dflare_config& c = h->cfg;
  const long D = c.n_draft_layers;
  const long lm = (long)ceil_div(c.vocab, 16) * (c.hidden / 32) * 64;
  struct Item {
    u32x4** dst;
    const u32x4* src;
    long n;
  } items[] = {{&h->h_qkv, h->w_qkv, h->s_qkv * D}, {&h->h_o, h->w_o, h->s_o * D},
               {&h->h_gu, h->w_gu, h->s_gu * D},    {&h->h_down, h->w_down, h->s_down * D},
               {&h->h_kvt, h->w_kvt, h->s_kvt * D}, {&h->h_lm, h->w_lm, lm}};
  for (const Item& it : items) {
    u32x4* p = nullptr;
    TRY(dev_alloc(h, &p, (size_t)it.n * 16));
    launch_tiles_to_f16(h->stream, p, it.src, it.n);
    *it.dst = p;
  }
  if (h->w_fc) {
    const long n = (long)(c.hidden / 16) * (c.n_target_layers * c.hidden / 32) * 64;
    TRY(dev_alloc(h, &h->h_fc, (size_t)n * 16));
    launch_tiles_to_f16(h->stream, h->h_fc, h->w_fc, n);
  }
  return check_launch(h, "weight conversion");
}

// one batched GEMM with its fused epilogue; the K split is chosen per shape
void bgemm(dflare_handle* h, int kind, const char* name, int epi, BGemmArgs g, const BRows& rows) {
  g.nw = bgemm_nw(h->cus, name, g.Nt, g.Mt, g.Kt, g.layers, epi != BEPI_ARGMAX && epi != BEPI_BIAS16);
  g.kg = bgemm_split(h->cus, name, g.Nt, g.Mt, g.Kt, g.layers, epi != BEPI_ARGMAX, g.nw);
  g.zero = h->zero_tile;
  g.part = h->bpart;
  g.cnt = h->bcnt;
  prof_mark(h, kind, true);
  launch_bgemm(h->stream, epi, g, rows);
  prof_mark(h, kind, false);
}

// epilogue fields shared by every batched GEMM of a handle
BGemmArgs bgemm_base(const dflare_handle* h) {
  const dflare_config& c = h->cfg;
  BGemmArgs g{};
  g.layers = 1;
  g.Q = h->bQ;
  g.q_dim = h->q_dim;
  g.kc = h->kc;
  g.vt = h->vt;
  g.seq_stride = h->seq_stride;
  g.cache_layer = h->cache_layer_stride;
  g.Lcap = h->Lcap;
  g.hd = c.head_dim;
  g.q_tiles = h->q_dim / 16;
  g.kv_tiles = h->kv_dim / 16;
  g.rope = h->rope;
  g.X = h->bX;
  g.H = c.hidden;
  g.out16 = h->bHA;
  g.out_kt = c.ffn / 32;
  g.V = c.vocab;
  g.pmax = h->bpmax;
  g.pidx = h->bpidx;
  g.pld = h->b_mt * 16;
  return g;
}

// hidden: [S, ld, H]; the call's rows are rows 0 .. sum(n_new) - 1 of each target layer
int run_fuse_batched(dflare_handle* h, int n_seq, const int32_t* seq, const int32_t* n_new, const void* hidden,
                     int ld) {
  const dflare_config& c = h->cfg;
  const int H = c.hidden, D = c.n_draft_layers, S = c.n_target_layers, Kt_H = H / 32;
  hipStream_t s = h->stream;
  BRows rows{};
  rows.n_seq = n_seq;
  for (int i = 0; i < n_seq; ++i) {
    rows.seq[i] = seq[i];
    rows.L[i] = h->Ls[seq[i]];
    rows.off[i + 1] = rows.off[i] + n_new[i];
  }
  const int N = rows.off[n_seq];
  const bool dflash = c.variant & DFLARE_VARIANT_DFLASH;
  BGemmArgs g = bgemm_base(h);
  if (dflash) {
    // Eq. 1: C = [h^(1); ...; h^(S)] W_fc^T + b_fc for all N rows, as fp16 fragments
    prof_mark(h, DFLARE_K_B_FUSE, true);
    launch_bfrag_cat(s, (const uint16_t*)hidden, N, ld, S, H, h->bCat);
    g.A = h->bCat;
    g.a_layer = 0;
    g.W = h->h_fc;
    g.w_layer = 0;
    g.Nt = H / 16;
    g.Kt = S * H / 32;
    g.Mt = ceil_div(N, 16);
    g.M = N;
    g.out16 = h->bC;
    g.out_kt = Kt_H;
    g.bias = h->fc_bias;
    bgemm(h, -1, "FC", BEPI_BIAS16, g, rows);
    prof_mark(h, DFLARE_K_B_FUSE, false);
    g = bgemm_base(h);
    g.A = h->bC;  // the same context rows for every layer (Eq. 2)
    g.a_layer = 0;
  } else {
    prof_mark(h, DFLARE_K_B_FUSE, true);
    launch_bfuse(s, (const uint16_t*)hidden, N, ld, S, H, D, h->alpha, h->g_fuse, c.rms_eps, h->bU, h->mt_max);
    prof_mark(h, DFLARE_K_B_FUSE, false);
    g.A = h->bU;
    g.a_layer = (long)h->mt_max * Kt_H * 64;
    g.bias = h->kv_bias;
  }
  g.W = h->h_kvt;
  g.w_layer = h->s_kvt;
  g.Nt = 2 * h->kv_dim / 16;
  g.Kt = Kt_H;
  g.Mt = ceil_div(N, 16);
  g.M = N;
  g.layers = D;
  g.layer0 = 0;
  g.q_tiles = 0;
  bgemm(h, DFLARE_K_B_KV_T, "KVT", BEPI_QKV, g, rows);
  if (h->debug) {  // DFlash: the shared context rows, as layer 0
    launch_bfrag_rows(s, dflash ? h->bC : h->bU, N, H, dflash ? 1 : D, h->mt_max, h->dbg_fused);
    h->dbg_fused_n = N;
  }
  TRY(check_launch(h, "fuse_append_batched"));
  for (int i = 0; i < n_seq; ++i) h->Ls[seq[i]] += n_new[i];
  return DFLARE_OK;
}

int run_draft_batched(dflare_handle* h, int n_seq, const int32_t* seq, const int32_t* ids, int32_t* out) {
  const dflare_config& c = h->cfg;
  const int H = c.hidden, F = c.ffn, V = c.vocab, D = c.n_draft_layers, B = c.block_size, hd = c.head_dim;
  const int Kt_H = H / 32, Kt_q = h->q_dim / 32, Kt_F = F / 32;
  const int Nt_qkv = (h->q_dim + 2 * h->kv_dim) / 16, Nt_H = H / 16, Nt_gu = 2 * F / 16, Nt_lm = ceil_div(V, 16);
  hipStream_t s = h->stream;
  const int M = n_seq * B, Mt = ceil_div(M, 16);
  BRows rows{};
  rows.n_seq = n_seq;
  for (int i = 0; i < n_seq; ++i) {
    rows.seq[i] = seq[i];
    rows.L[i] = h->Ls[seq[i]];
    rows.off[i + 1] = (i + 1) * B;
    rows.ipfx[i + 1] = rows.ipfx[i] + ceil_div(rows.L[i] + B, kBKeys) * c.n_kv_heads;
  }
  const int items = rows.ipfx[n_seq];
  BAttnArgs at{};
  at.Q = h->bQ;
  at.kc = h->kc;
  at.vt = h->vt;
  at.seq_stride = h->seq_stride;
  at.cache_layer = h->cache_layer_stride;
  at.Lcap = h->Lcap;
  at.B = B;
  at.n_q = c.n_q_heads;
  at.n_kv = c.n_kv_heads;
  at.Rpad = h->Rpad;
  at.qscale = (float)(1.4426950408889634 / sqrt((double)hd));
  at.OP = h->bOP;
  at.ML = h->bML;
  BGemmArgs g = bgemm_base(h);
  g.Mt = Mt;
  g.M = M;

  prof_mark(h, DFLARE_K_B_EPI, true);
  launch_bembed_norm(s, h->embed, ids, M, H, V, h->g_attn, c.rms_eps, h->bX, h->bA, Kt_H);
  prof_mark(h, DFLARE_K_B_EPI, false);
  for (int l = 0; l < D; ++l) {
    g.layer0 = l;
    g.A = h->bA;
    g.W = h->h_qkv + l * h->s_qkv;
    g.Nt = Nt_qkv;
    g.Kt = Kt_H;
    bgemm(h, DFLARE_K_B_QKV, "QKV", BEPI_QKV, g, rows);
    at.layer = l;
    prof_mark(h, DFLARE_K_B_ATTN, true);
    launch_battn(s, hd, at, rows, items);
    launch_bcomb(s, hd, at, rows, h->bOA, Kt_q);
    prof_mark(h, DFLARE_K_B_ATTN, false);
    g.A = h->bOA;
    g.W = h->h_o + l * h->s_o;
    g.Nt = Nt_H;
    g.Kt = Kt_q;
    bgemm(h, DFLARE_K_B_O, "O", BEPI_RESID, g, rows);
    prof_mark(h, DFLARE_K_B_EPI, true);
    launch_bnorm(s, h->bX, M, H, h->g_mlp + (long)l * H, c.rms_eps, h->bA, Kt_H);
    prof_mark(h, DFLARE_K_B_EPI, false);
    g.A = h->bA;
    g.W = h->h_gu + l * h->s_gu;
    g.Nt = Nt_gu;
    g.Kt = Kt_H;
    bgemm(h, DFLARE_K_B_GATE_UP, "GU", BEPI_SWIGLU, g, rows);
    g.A = h->bHA;
    g.W = h->h_down + l * h->s_down;
    g.Nt = Nt_H;
    g.Kt = Kt_F;
    bgemm(h, DFLARE_K_B_DOWN, "DOWN", BEPI_RESID, g, rows);
    prof_mark(h, DFLARE_K_B_EPI, true);
    launch_bnorm(s, h->bX, M, H, (l + 1 < D) ? h->g_attn + (long)(l + 1) * H : h->g_final, c.rms_eps, h->bA, Kt_H);
    prof_mark(h, DFLARE_K_B_EPI, false);
  }
  g.A = h->bA;
  g.W = h->h_lm;
  g.Nt = Nt_lm;
  g.Kt = Kt_H;
  g.logits = h->debug ? h->dbg_blogits : nullptr;
  g.inv_temp = h->temperature > 0.f ? 1.0f / h->temperature : 0.f;
  g.draw = h->draw;
  g.seed = h->seed;
  if (h->temperature > 0.f) ++h->draw;
  prof_mark(h, DFLARE_K_B_LM_HEAD, true);
  bgemm(h, -1, "LM", BEPI_ARGMAX, g, rows);  // timed with the final argmax below
  launch_bargmax(s, h->bpmax, h->bpidx, ceil_div(Nt_lm, kBN), g.pld, M, out);
  prof_mark(h, DFLARE_K_B_LM_HEAD, false);
  if (h->debug) h->dbg_blogits_rows = M;
  return check_launch(h, "draft_block_batched");
}

}  // namespace

extern "C" {

int dflare_init(const dflare_config* cfg, const dflare_weights* w, const float* fusion_logits, void* stream,
                dflare_handle** out) {
  g_init_error.clear();
  if (!out) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  TRY(validate_config(cfg));
  const int var = cfg->variant;
  const bool dflash = var & DFLARE_VARIANT_DFLASH;
  const bool need_t = !(var & (DFLARE_VARIANT_SHARED_KV | DFLARE_VARIANT_DFLASH));
  if (!w || !w->embed || !w->lm_head || !w->wq || !w->wk_d || !w->wv_d || (need_t && (!w->wk_t || !w->wv_t)) ||
      !w->wo || !w->w_gate || !w->w_up || !w->w_down)
    return fail(nullptr, DFLARE_ERR_INVALID_ARG, "a required weight pointer is NULL");
  if ((var & DFLARE_VARIANT_POST_FC) && !w->post_fc)
    return fail(nullptr, DFLARE_ERR_INVALID_ARG, "POST_FC needs post_fc");
  if (dflash && !w->fc) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "DFLASH needs fc");
  if (!fusion_logits && !dflash) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "fusion_logits is NULL");
  const int D = cfg->n_draft_layers, S = cfg->n_target_layers;
  // alpha^(i) = softmax(W^fuse_{i,:}) in double precision, cached as float (Sec. 4.1);
  // -Softmax (Sec. 6.3) keeps W^fuse itself; DFlash has no fusion weights
  std::vector<float> alpha((size_t)D * S, 0.f);
  for (int i = 0; i < D && !dflash; ++i) {
    if (var & DFLARE_VARIANT_NO_SOFTMAX) {
      for (int j = 0; j < S; ++j) {
        const float x = fusion_logits[(size_t)i * S + j];
        if (!isfinite(x)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "unnormalised fusion weights must be finite");
        alpha[(size_t)i * S + j] = x;
      }
      continue;
    }
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
  if (h->cfg.max_batch == 0) h->cfg.max_batch = 1;
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

// Append rows 0 .. n_new-1 of target_hidden [S, ld, H] to slot 0 (arguments validated).
// With Lp the rows go to slots *Lp + row, and the host's length is left alone.
int append_rows(dflare_handle* h, const void* target_hidden, int32_t n_new, int ld, const int32_t* Lp = nullptr) {
  const dflare_config& c = h->cfg;
  if (c.variant & DFLARE_VARIANT_DFLASH) {  // the FC fusion runs on the batched GEMM, slot 0
    const int32_t seq0 = 0;
    return run_fuse_batched(h, 1, &seq0, &n_new, target_hidden, ld);
  }
  const int H = c.hidden, D = c.n_draft_layers, S = c.n_target_layers;
  hipStream_t s = h->stream;
  prof_mark(h, DFLARE_K_FUSE, true);
  launch_fuse(s, (const uint16_t*)target_hidden, n_new, ld, S, H, D, h->alpha, h->g_fuse, h->Ustats, h->ua_hi,
              h->ua_lo, c.max_new, h->mt_max);
  prof_mark(h, DFLARE_K_FUSE, false);
  KvtArgs a{};
  a.W = h->w_kvt;
  a.w_layer_stride = h->s_kvt;
  a.Nt = 2 * h->kv_dim / 16;
  a.Kt = H / 32;
  a.zero = h->zero_tile;
  a.Ahi = h->ua_hi;
  a.Alo = h->ua_lo;
  a.a_layer_stride = (long)h->mt_max * (H / 32) * 64;
  a.stats = h->Ustats;
  a.stats_layer_stride = (long)c.max_new * (H / 16);
  a.n_stat = H / 16;
  a.inv_dim = 1.0f / H;
  a.eps = c.rms_eps;
  a.L = Lp ? 0 : h->Ls[0];
  a.Lp = Lp;
  a.n_new = n_new;
  a.kc = h->kc;
  a.vt = h->vt;
  a.cache_layer_stride = h->cache_layer_stride;
  a.Lcap = h->Lcap;
  a.hd = c.head_dim;
  a.kv_tiles = h->kv_dim / 16;
  a.rope = h->rope;
  a.bias = h->kv_bias;
  prof_mark(h, DFLARE_K_KV_T, true);
  launch_kvt(s, h->kvt_nt, h->kvt_waves, a, D, ceil_div(n_new, 16));
  prof_mark(h, DFLARE_K_KV_T, false);
  if (h->debug) {
    launch_fused_rows(s, h->ua_hi, h->ua_lo, h->Ustats, n_new, H, D, c.max_new, h->mt_max, c.rms_eps,
                      h->dbg_fused);
    h->dbg_fused_n = n_new;
  }
  int rc = check_launch(h, "fuse_append");
  if (rc != DFLARE_OK) return rc;
  if (!Lp) h->Ls[0] += n_new;
  return DFLARE_OK;
}


int dflare_fuse_append(dflare_handle* h, const void* target_hidden, int32_t n_new) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  TRY(settle_len(h));
  if (!target_hidden) return fail(h, DFLARE_ERR_INVALID_ARG, "target_hidden is NULL");
  if (n_new < 1 || n_new > h->cfg.max_new)
    return fail(h, DFLARE_ERR_INVALID_ARG, "n_new must be in [1, max_new]");
  if ((long)h->Ls[0] + n_new > h->cfg.max_context)
    return fail(h, DFLARE_ERR_CONTEXT_FULL, "append would exceed max_context");
  return append_rows(h, target_hidden, n_new, n_new);
}

int dflare_accept(dflare_handle* h, const int32_t* block_ids, const int32_t* draft_tokens, const int32_t* target_tokens,
                  const void* target_hidden, int32_t* next_ids, int32_t* emitted, int32_t* accepted) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  TRY(settle_len(h));
  if (!block_ids || !draft_tokens || !target_tokens || !target_hidden || !next_ids || !emitted)
    return fail(h, DFLARE_ERR_INVALID_ARG, "a device pointer is NULL");
  const dflare_config& c = h->cfg;
  const int B = c.block_size;
  if (c.max_new < B) return fail(h, DFLARE_ERR_INVALID_ARG, "dflare_accept needs max_new >= block_size");
  if ((long)h->Ls[0] + B > c.max_context)
    return fail(h, DFLARE_ERR_CONTEXT_FULL, "a verified block could exceed max_context");
  int32_t* k_host = h->err_host + 8;  // host-mapped word next to the barrier flag
  int32_t* k_dev = h->err_dev + 8;
  *(volatile int32_t*)k_host = -1;
  launch_accept(h->stream, block_ids, draft_tokens, target_tokens, B, next_ids, emitted, k_dev, nullptr, 0, nullptr);
  TRY(check_launch(h, "accept"));
  HIP_OR_FAIL(h, hipStreamSynchronize(h->stream));
  const int k = *(volatile int32_t*)k_host;
  if (k < 0 || k >= B) return fail(h, DFLARE_ERR_HIP, "verification result not received");
  TRY(append_rows(h, target_hidden, k + 1, B));
  if (accepted) *accepted = k;
  return DFLARE_OK;
}

int dflare_accept_async(dflare_handle* h, const int32_t* block_ids, const int32_t* draft_tokens,
                        const int32_t* target_tokens, const void* target_hidden, int32_t* next_ids,
                        int32_t* emitted, int32_t* accepted_dev) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  if (!block_ids || !draft_tokens || !target_tokens || !target_hidden || !next_ids || !emitted)
    return fail(h, DFLARE_ERR_INVALID_ARG, "a device pointer is NULL");
  const dflare_config& c = h->cfg;
  const int B = c.block_size;
  if (c.max_new < B) return fail(h, DFLARE_ERR_INVALID_ARG, "dflare_accept_async needs max_new >= block_size");
  if (c.variant & DFLARE_VARIANT_DFLASH) {  // its fusion runs on the batched path, which takes host lengths
    int32_t k = 0;
    TRY(dflare_accept(h, block_ids, draft_tokens, target_tokens, target_hidden, next_ids, emitted, &k));
    if (accepted_dev) {
      HIP_OR_FAIL(h, hipMemcpyAsync(accepted_dev, &k, sizeof(k), hipMemcpyHostToDevice, h->stream));
      HIP_OR_FAIL(h, hipStreamSynchronize(h->stream));
    }
    return DFLARE_OK;
  }
  if (!h->dev_len) h->L_hi = h->Ls[0];
  if (h->L_hi + B > c.max_context) {  // the bound is too loose to promise room: look at the length itself
    TRY(settle_len(h));
    h->L_hi = h->Ls[0];
    if (h->L_hi + B > c.max_context)
      return fail(h, DFLARE_ERR_CONTEXT_FULL, "a verified block could exceed max_context");
  }
  const int32_t* Lp = h->dev_len ? h->Ldev + h->lcur : nullptr;
  launch_accept(h->stream, block_ids, draft_tokens, target_tokens, B, next_ids, emitted,
                accepted_dev ? accepted_dev : h->kdev, Lp, h->Ls[0], h->Ldev + (h->lcur ^ 1));
  TRY(check_launch(h, "accept"));
  // all B rows go to slots L .. L + B - 1; the ones past the k + 1 verified rows lie beyond
  // the new length, where the next draft block writes its own keys before anything reads them
  const int32_t L_now = h->Ls[0];
  const int32_t* base = Lp;
  if (!base) {  // first step with the length on the device: the host value is still exact
    TRY(append_rows(h, target_hidden, B, B));
    h->Ls[0] = L_now;
  } else {
    TRY(append_rows(h, target_hidden, B, B, base));
  }
  h->lcur ^= 1;
  h->dev_len = true;
  h->L_hi += B;
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
  TRY(settle_len(h));
  if (!block_ids || !draft_tokens || !positions)
    return fail(h, DFLARE_ERR_INVALID_ARG, "block_ids / positions / draft_tokens is NULL");
  for (int b = 0; b < h->cfg.block_size; ++b)
    if (positions[b] < 0 || positions[b] >= h->cfg.max_context + h->cfg.block_size)
      return fail(h, DFLARE_ERR_INVALID_ARG, "a position is outside [0, max_context + block_size)");
  return run_draft_block(h, block_ids, positions, draft_tokens);
}

int dflare_fuse_append_batched(dflare_handle* h, int32_t n_seq, const int32_t* seq, const int32_t* n_new,
                               const void* target_hidden) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  TRY(check_seqs(h, n_seq, seq));
  if (!n_new || !target_hidden) return fail(h, DFLARE_ERR_INVALID_ARG, "n_new / target_hidden is NULL");
  long total = 0;
  for (int i = 0; i < n_seq; ++i) {
    if (n_new[i] < 1) return fail(h, DFLARE_ERR_INVALID_ARG, "every n_new must be >= 1");
    total += n_new[i];
  }
  if (total > h->cfg.max_new) return fail(h, DFLARE_ERR_INVALID_ARG, "sum of n_new must be <= max_new");
  for (int i = 0; i < n_seq; ++i)
    if ((long)h->Ls[seq[i]] + n_new[i] > h->cfg.max_context)
      return fail(h, DFLARE_ERR_CONTEXT_FULL, "append would exceed max_context");
  TRY(ensure_f16_weights(h));
  prof_mark(h, DFLARE_K_B_APPEND, true);
  const int rc = run_fuse_batched(h, n_seq, seq, n_new, target_hidden, (int)total);
  prof_mark(h, DFLARE_K_B_APPEND, false);
  return rc;
}

int dflare_draft_block_batched(dflare_handle* h, int32_t n_seq, const int32_t* seq, const int32_t* block_ids,
                               int32_t* draft_tokens) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  TRY(check_seqs(h, n_seq, seq));
  if (!block_ids || !draft_tokens) return fail(h, DFLARE_ERR_INVALID_ARG, "block_ids / draft_tokens is NULL");
  TRY(ensure_f16_weights(h));
  prof_mark(h, DFLARE_K_B_DRAFT, true);
  const int rc = run_draft_batched(h, n_seq, seq, block_ids, draft_tokens);
  prof_mark(h, DFLARE_K_B_DRAFT, false);
  return rc;
}

int dflare_set_sampling(dflare_handle* h, float temperature, uint64_t seed) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  if (!(temperature >= 0.f) || !isfinite(temperature) || (temperature > 0.f && !isfinite(1.f / temperature)))
    return fail(h, DFLARE_ERR_INVALID_ARG, "temperature must be 0 or finite with a finite reciprocal");
  h->temperature = temperature;
  h->seed = seed;
  h->draw = 0;
  return DFLARE_OK;
}

int dflare_truncate_seq(dflare_handle* h, int32_t seq, int32_t new_len) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  TRY(settle_len(h));
  if (seq < 0 || seq >= h->cfg.max_batch) return fail(h, DFLARE_ERR_INVALID_ARG, "seq must be in [0, max_batch)");
  if (new_len < 0 || new_len > h->Ls[seq]) return fail(h, DFLARE_ERR_INVALID_ARG, "new_len must be in [0, L]");
  h->Ls[seq] = new_len;
  return DFLARE_OK;
}

int dflare_context_len_seq(const dflare_handle* h, int32_t seq, int32_t* out) {
  if (!live(h) || !out || seq < 0 || seq >= h->cfg.max_batch) return DFLARE_ERR_INVALID_ARG;
  if (seq == 0 && settle_len(const_cast<dflare_handle*>(h)) != DFLARE_OK) return DFLARE_ERR_HIP;
  *out = h->Ls[seq];
  return DFLARE_OK;
}

int dflare_truncate(dflare_handle* h, int32_t new_len) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  TRY(settle_len(h));
  if (new_len < 0 || new_len > h->Ls[0]) return fail(h, DFLARE_ERR_INVALID_ARG, "new_len must be in [0, L]");
  h->Ls[0] = new_len;
  return DFLARE_OK;
}

int dflare_context_len(const dflare_handle* h, int32_t* out) {
  if (!live(h) || !out) return DFLARE_ERR_INVALID_ARG;
  if (settle_len(const_cast<dflare_handle*>(h)) != DFLARE_OK) return DFLARE_ERR_HIP;
  *out = h->Ls[0];
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
    TRY(dev_alloc(h, &h->dbg_blogits, (size_t)c.max_batch * c.block_size * c.vocab * 4));
  }
  h->debug = on != 0;
  return DFLARE_OK;
}

int dflare_debug_read(dflare_handle* h, int what, int layer, float* host_out, int64_t count) {
  return dflare_debug_read_seq(h, what, 0, layer, host_out, count);
}

int dflare_debug_read_seq(dflare_handle* h, int what, int seq, int layer, float* host_out, int64_t count) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  TRY(settle_len(h));
  if (!host_out) return fail(h, DFLARE_ERR_INVALID_ARG, "host_out is NULL");
  if (seq < 0 || seq >= h->cfg.max_batch) return fail(h, DFLARE_ERR_INVALID_ARG, "seq must be in [0, max_batch)");
  if (seq != 0 && what != DFLARE_DBG_KCACHE && what != DFLARE_DBG_VCACHE)
    return fail(h, DFLARE_ERR_INVALID_ARG, "only the caches are read per sequence slot");
  const dflare_config& c = h->cfg;
  const int H = c.hidden, B = c.block_size, hd = c.head_dim, nkv = c.n_kv_heads;
  const bool needs_layer = what == DFLARE_DBG_FUSED || what == DFLARE_DBG_KCACHE || what == DFLARE_DBG_VCACHE ||
                           what == DFLARE_DBG_HIDDEN;
  if (needs_layer && (layer < 0 || layer >= c.n_draft_layers))
    return fail(h, DFLARE_ERR_INVALID_ARG, "layer out of range");
  if ((what == DFLARE_DBG_FUSED || what == DFLARE_DBG_HIDDEN || what == DFLARE_DBG_LOGITS ||
       what == DFLARE_DBG_BLOGITS) && !h->dbg_hidden)
    return fail(h, DFLARE_ERR_INVALID_ARG, "debug capture was never enabled");
  if (what == DFLARE_DBG_TRACE && !h->trace_buf) return fail(h, DFLARE_ERR_INVALID_ARG, "tracing was never enabled");
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
    case DFLARE_DBG_BLOGITS: {
      const int64_t n = (int64_t)h->dbg_blogits_rows * c.vocab;
      if (count < n) return fail(h, DFLARE_ERR_INVALID_ARG, "host buffer too small");
      HIP_OR_FAIL(h, hipMemcpy(host_out, h->dbg_blogits, n * 4, hipMemcpyDeviceToHost));
      return DFLARE_OK;
    }
    case DFLARE_DBG_KCACHE:
    case DFLARE_DBG_VCACHE: {
      const int L = h->Ls[seq];
      const int64_t n = (int64_t)L * nkv * hd;
      if (count < n) return fail(h, DFLARE_ERR_INVALID_ARG, "host buffer too small");
      std::vector<uint16_t> raw((size_t)h->cache_layer_stride);
      const uint16_t* src = (what == DFLARE_DBG_KCACHE ? h->kc : h->vt) + seq * h->seq_stride +
                            (long)layer * h->cache_layer_stride;
      HIP_OR_FAIL(h, hipMemcpy(raw.data(), src, raw.size() * 2, hipMemcpyDeviceToHost));
      for (int p = 0; p < L; ++p)
        for (int g = 0; g < nkv; ++g)
          for (int d = 0; d < hd; ++d) {
            const size_t ix = (what == DFLARE_DBG_KCACHE) ? ((size_t)g * h->Lcap + p) * hd + d
                                                          : ((size_t)g * hd + d) * h->Lcap + p;
            host_out[((size_t)p * nkv + g) * hd + d] = half_to_float(raw[ix]);
          }
      return DFLARE_OK;
    }
    case DFLARE_DBG_TRACE: {
      const int64_t n = (int64_t)h->blocks * kTraceSlots * h->phases;
      if (count < n) return fail(h, DFLARE_ERR_INVALID_ARG, "host buffer too small");
      std::vector<unsigned long long> raw((size_t)n);
      HIP_OR_FAIL(h, hipMemcpy(raw.data(), h->trace_buf, n * 8, hipMemcpyDeviceToHost));
      unsigned long long t0 = ~0ull;
      for (int64_t i = 0; i < n; ++i)
        if (raw[i]) t0 = std::min(t0, raw[i]);
      for (int64_t i = 0; i < n; ++i)  // 100 MHz ticks -> us; marks a phase does not set: -1
        host_out[i] = raw[i] ? (float)((double)(raw[i] - t0) * 0.01) : -1.0f;
      return DFLARE_OK;
    }
    default: return fail(h, DFLARE_ERR_INVALID_ARG, "unknown debug tensor");
  }
}

int dflare_profile_begin(dflare_handle* h, int kind) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  if (kind < 0 || kind > DFLARE_K_B_APPEND) return fail(h, DFLARE_ERR_INVALID_ARG, "unknown kernel kind");
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
  const int32_t v[6] = {h->persistent ? 1 : h->phases, 2, h->blocks, h->phases,
                        h->persistent ? h->phases - 1 - 2 * h->cfg.n_draft_layers : 0,
                        h->generic_draft ? 0 : h->draft_sig};
  for (int i = 0; i < count && i < 6; ++i) out[i] = v[i];
  return DFLARE_OK;
}

int dflare_read_probe(const void* buf, int64_t bytes, uint32_t* sink, void* stream) {
  if (!buf || !sink || bytes <= 0 || bytes % 16) return DFLARE_ERR_INVALID_ARG;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return DFLARE_ERR_HIP;
  launch_read_probe((hipStream_t)stream, buf, (long)bytes, sink, 8 * cus);
  return hipGetLastError() == hipSuccess ? DFLARE_OK : DFLARE_ERR_HIP;
}

int dflare_set_option(dflare_handle* h, int option, int value) {
  if (!live(h)) return fail(nullptr, DFLARE_ERR_INVALID_ARG, "invalid handle");
  switch (option) {
    case DFLARE_OPT_PERSISTENT:
      if (value && !h->coop_ok)
        return fail(h, DFLARE_ERR_UNSUPPORTED, "the device cannot keep one draft work-group per CU resident");
      h->persistent = value != 0;
      return DFLARE_OK;
    case DFLARE_OPT_TRACE:
      h->trace = value != 0;
      return DFLARE_OK;
    case DFLARE_OPT_CAPTURE_PERSISTENT:
      h->capture_persistent = value != 0;
      return DFLARE_OK;
    case DFLARE_OPT_COOPERATIVE:
      h->coop_launch = value != 0;
      return DFLARE_OK;
    case DFLARE_OPT_GENERIC_KERNEL:
      h->generic_draft = value != 0;
      return DFLARE_OK;
    default: return fail(h, DFLARE_ERR_INVALID_ARG, "unknown option");
  }
}

}  // extern "C"
