// Internal declarations shared by the kernel and runtime translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dflare {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Every weight matrix W[N, K] (y = x W^T) is re-packed at init into 16 x 32
// tiles, one per (n-tile, k-tile), stored n-tile major:
//   tile (nt, kt) = 64 lanes x 16 bytes at ((nt * Kt + kt) * 64 + lane);
//   lane l holds W[row(nt*16 + l%16)][kt*32 + 8*(l/16) .. +7]
// which is exactly the B operand of v_mfma_f32_16x16x32_bf16, so one wave reads a
// tile with a single fully coalesced 1 KiB load.  row() permutes output rows:
enum PackMode {
  PACK_IDENTITY = 0,  // row(p) = p
  PACK_ROPE = 1,      // each 16-column tile holds 8 rotary pairs (m, m + hd/2)
  PACK_SWIGLU = 2     // each 16-column tile holds 8 gate rows then the 8 matching up rows
};

constexpr int kThreads = 512;   // draft-block work-group: 8 waves, one work-group per CU
constexpr int kWaves = kThreads / 64;
constexpr int kStatsPad = 32;   // floats per 16-column tile in the sums-of-squares arrays (one 128 B line)
constexpr int kBarCounters = 16;  // grid-barrier arrival counters, each on its own 128 B line
constexpr int kMaxBlock = 16;     // draft block rows (one 16-row MFMA tile)
constexpr int kChunk = 128;       // context keys per attention work item
// wall-clock marks per phase: body start (after the grid barrier), two inner marks
// (GEMM: main loop done, chunk epilogues done; attention: keys staged, scores and
// values done; combine: partials loaded), stores complete
constexpr int kTraceSlots = 4;
constexpr int kTNMax = 8;         // output tiles a GEMM work-group accumulates at once
constexpr int kMaxSplit = 8;      // work-groups that split one GEMM output range along K
constexpr int kMaxBlocks = 1024;  // work-groups of the draft-block kernel
// GEMM phase kinds that may split K (one tagged partial area each); a reserved block of
// kSplitKinds x kMaxBlocks counter lines follows the grid-barrier counters and the LM-head
// completion counter in the synchronisation area.
constexpr int kSplitKinds = 4;    // QKV, O, gate/up, down
// Attention arrival counters, then Q/K/V tile counters: one per KV head each, each on its own
// 128 B line, after the split-K ones.
constexpr int kMaxKvHeads = 128;
constexpr long kAttnCntOff = 4096 + (long)kSplitKinds * kMaxBlocks * 128;  // bytes
constexpr long kQkvCntOff = kAttnCntOff + (long)kMaxKvHeads * 128;         // bytes
constexpr long kSyncBytes = kQkvCntOff + (long)kMaxKvHeads * 128;
// Zero k-tiles after the K real ones in every draft-block activation (A-fragment) plane:
// a GEMM wave's run of k-tiles may reach past K, by less than 2 * 8 + 1 batches of 4.
constexpr int kKtPad = 72;
// Spare bytes after every packed weight matrix: the last batch of a row may reach past K.
constexpr long kWeightSpare = 64 * 1024;

// The draft block is one sequence of phases; between two phases every work-group waits
// at a grid barrier (one persistent launch) or the phases are separate launches.
//   EMBED, then for each draft layer QKV, ATTN, COMB, O, GU, DOWN, then LM.
enum Phase { PH_EMBED = 0, PH_QKV, PH_ATTN, PH_COMB, PH_O, PH_GU, PH_DOWN, PH_LM, PH_COUNT };
__host__ __device__ inline int phase_count(int D) { return 2 + 6 * D; }
__host__ __device__ inline void phase_of(int p, int D, int& kind, int& layer) {
  if (p == 0) {
    kind = PH_EMBED;
    layer = 0;
  } else if (p == 1 + 6 * D) {
    kind = PH_LM;
    layer = D;
  } else {
    kind = PH_QKV + (p - 1) % 6;
    layer = (p - 1) / 6;
  }
}

// What changes from one draft block to the next: passed by value at every launch.
struct DraftCall {
  int L;                // context length (when Lp is NULL)
  const int* Lp;        // device-resident context length, or NULL: then L above
  int pos[kMaxBlock];   // positions of the block rows (with Lp: offsets added to *Lp)
  const int* ids;       // [B] block token ids
  int* tokens;          // [B] output: greedy draft tokens
  float* logits;        // optional [B, V]
  float* hidden;        // optional [D, B, H]: block rows after each draft layer
  unsigned bar_epoch;   // grid barriers completed by earlier launches
  unsigned done_epoch;  // launches that ran the LM phase before this one
  unsigned acnt_base;   // value of every attention arrival counter before this launch
  unsigned qcnt_base;   // value of every Q/K/V tile counter before this launch
  unsigned long long* trace;  // optional [blocks][phases][kTraceSlots] wall clock at marks of each phase
  // candidate selection: inv_temp = 0 greedy argmax; otherwise argmax of z * inv_temp plus
  // Gumbel noise of draw `draw` under `seed` (sequence slot 0)
  float inv_temp;
  unsigned draw;
  unsigned long long seed;
};

// Everything else the draft-block kernel needs; written to device memory once at init and
// read through a pointer, so that the kernel loads each field where a phase uses it instead
// of holding all of them in scalar registers for the whole launch.  Data that one phase
// hands to a later one is written with write-through (agent-coherent) stores and is either
// written once per launch (per-stage and per-layer buffers, read with ordinary cached
// loads) or read back with coherent loads (the residual stream, the attention partials,
// the LM-head partial maxima); see the kernel source for the rule.
struct DraftArgs {
  // shapes
  // nch: attention chunks per layer the partial buffers hold (context keys per chunk: 128 at
  // head size 128, 256 at head size 64)
  int H, F, V, D, B, hd, n_q, n_kv, Lcap, Rpad, chunk, nch;
  float eps, qscale;
  // GEMM plan of each phase kind: the work-groups form blocks / kg output ranges of
  // consecutive n-tiles, kg work-groups per range each taking 1/kg of K; a work-group
  // accumulates up to tn (2, 3, 4, 5, 6 or 8) n-tiles at once.
  int tn[PH_COUNT], kg[PH_COUNT];
  // the partition, precomputed: output range r holds nq + (r < nr) n-tiles starting at
  // r * nq + min(r, nr); K part k holds kq + (k < kr) k-tiles starting at k * kq + min(k, kr)
  int nq[PH_COUNT], nr[PH_COUNT], kq[PH_COUNT], kr[PH_COUNT];
  // weights: packed tiles; strides between layers in u32x4 units
  const uint16_t* embed;
  const u32x4 *w_qkv, *w_o, *w_gu, *w_down, *w_lm;
  long s_qkv, s_o, s_gu, s_down;
  const float *g_attn, *g_mlp, *g_final;  // RMSNorm gains [D, H], [D, H], [H]
  const u32x4* zero;                      // one zero tile
  const float2* rope;                     // [Lcap, hd/2] (cos, sin)
  // context cache of layer 0 (fp16): K [n_kv, Lcap, hd], V^T [n_kv, hd, Lcap]
  uint16_t *kc, *vt;
  long cache_layer;
  // activations
  float* X;              // residual stream [16, H] fp32, updated in place
  float* XS;             // per stage: sums of squares [H/16][kStatsPad]
  long xs_stride;
  u32x4* XA;             // per stage: A fragments of x * gain, hi plane then lo plane (K + kKtPad k-tiles each)
  long xa_stride;
  float* Q;              // per layer: rotated queries [16, q_dim]
  long q_stride;
  uint16_t* OP;          // attention partials [D, nch, n_kv, G * 16, hd] fp16, divided by their sums
                         // (row t*16 + b: query head t of the KV head, block position b)
  float2* ML;            // [D, nch, n_kv, G * 16] (running max, sum), log2 domain
  u32x4* OA;             // per layer: A fragments of the attention output
  long oa_stride;
  u32x4* HA;             // per layer: A fragments of the SwiGLU output
  long ha_stride;
  float* pmax;           // [blocks][kStatsPad] best logit of each work-group per row
  int* pidx;
  float* part;           // split-K partial sums [kSplitKinds][blocks][kTNMax][64 lanes][4], tagged per use
  unsigned* kcnt;        // spare counters [kSplitKinds][kMaxBlocks], 32 words apart (unused by the draft block)
  unsigned* acnt;        // attention arrival counters [n_kv], 32 words apart, monotonic across launches
  unsigned* qcnt;        // Q/K/V tile counters [n_kv], 32 words apart, monotonic across launches
  // synchronisation
  unsigned* bar;          // kBarCounters counters, 32 words apart, monotonic across launches
  unsigned* done;         // LM-head completion counter, monotonic across launches
  int* err;               // host-mapped flag, set when a grid barrier times out
};

// The draft kernel's one argument: phases [p0, p1) of a draft block.
struct DraftKernArgs {
  const DraftArgs* a;  // device copy of the fixed arguments
  DraftCall c;
  int p0, p1;
};

// Arguments of the context K/V projection of fuse_append (Eq. 4, W^t): fused rows of every
// draft layer -> RoPE(K) and V written into cache slots L .. L + n_new - 1.
struct KvtArgs {
  const u32x4* W;          // packed [K^t ; V^t] tiles of layer 0
  long w_layer_stride;
  int Nt, Kt;
  const u32x4* zero;
  const u32x4* Ahi;        // A fragments of u * g_fuse, [D][mt_max][Kt][64]
  const u32x4* Alo;
  long a_layer_stride;
  const float* stats;      // sums of squares [D][max_new][H/16]
  long stats_layer_stride;
  int n_stat;
  float inv_dim, eps;
  int L, n_new;
  const int* Lp;           // device-resident context length, or NULL: then L (rows go to slots L + row)
  uint16_t *kc, *vt;
  long cache_layer_stride;
  int Lcap, hd, kv_tiles;
  const float2* rope;
  const float* bias;       // optional fp32 [D][K kv | V kv], added before the rotation
};

// ---- launchers (kernels.hip) ----
void launch_pack(hipStream_t s, u32x4* dst, const uint16_t* src0, const uint16_t* src1,
                 int n_src_rows, int K, int nt_begin, int nt_count, int Kt_total, int mode, int hd);
void launch_bf16_to_f32(hipStream_t s, float* dst, const uint16_t* src, long n);
// init: out[R, K] (bf16, round to nearest even) = A[R, O] B[O, K] with bf16 row-major
// inputs, accumulated in double precision
void launch_compose(hipStream_t s, uint16_t* out, const uint16_t* A, const uint16_t* B, int R, int O, int K);
// init: y[R] (fp32) = A[R, O] b[O] in double precision (b bf16; NULL gives zeros)
void launch_matvec(hipStream_t s, float* y, const uint16_t* A, const uint16_t* b, int R, int O);
void launch_fuse(hipStream_t s, const uint16_t* hidden, int n, int ld, int S, int H, int D, const float* alpha,
                 const float* gain, float* ustats, u32x4* ua_hi, u32x4* ua_lo, int n_max, int mt_max);
// verification (Sec. 3.2): accepted count k (to host-visible memory), next block, emitted tokens
// L_next (optional): receives L + k + 1, L being *Lp or, with Lp NULL, L_imm
void launch_accept(hipStream_t s, const int32_t* block_ids, const int32_t* draft, const int32_t* target, int B,
                   int32_t* next_ids, int32_t* emitted, int32_t* k_out, const int32_t* Lp, int L_imm,
                   int32_t* L_next);
void launch_fused_rows(hipStream_t s, const u32x4* ua_hi, const u32x4* ua_lo, const float* ustats, int n,
                       int H, int D, int n_max, int mt_max, float eps, float* out);
bool kvt_shape_supported(int nt_per_block, int waves);
void launch_kvt(hipStream_t s, int nt_per_block, int waves, const KvtArgs& a, int layers, int mtiles);
// Phases [p0, p1) of a draft block on `blocks` work-groups of kThreads threads, which wait at
// grid barriers between phases (p1 > p0 + 1 needs all of them resident: one per CU, placed
// at once when no other stream holds CUs).  cooperative = true asks the runtime to
// guarantee that co-residency.  sig is the plans' signature (chunk widths of Q/K/V, output,
// gate/up and down, 4 bits each, draft_plan_sig): a kernel built for those plans runs if
// there is one, else the generic kernel (sig 0), with the same results.
hipError_t launch_draft(hipStream_t s, const DraftArgs* a_dev, const DraftCall& c, int hd, int sig, int blocks,
                        int p0, int p1, bool cooperative);
bool draft_specialized(int hd, int sig);
int draft_blocks_per_cu(int hd, int sig);
inline int draft_plan_sig(int tn_qkv, int tn_o, int tn_gu, int tn_down) {
  return tn_qkv | tn_o << 4 | tn_gu << 8 | tn_down << 12;
}
// measurement: streaming read of `bytes` (a multiple of 16) on `blocks` work-groups of 256
void launch_read_probe(hipStream_t s, const void* buf, long bytes, uint32_t* sink, int blocks);

}  // namespace dflare
