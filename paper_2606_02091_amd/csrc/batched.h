// Declarations of the batched draft step (batched.hip): many sequences, each with its own
// context cache, drafted together so that every projection is a GEMM over all their
// block rows.
#pragma once

#include "dflare_impl.h"

namespace dflare {

constexpr int kBWaves = 4;               // GEMM work-group: 4 waves
constexpr int kBWavesPerSimd = 2;        // GEMM work-groups resident per CU (waves per SIMD)
constexpr int kBPrefetch = 3;            // k-tiles of GEMM operand loads in flight per wave
constexpr int kBM = 8;                   // m-tiles per work-group (128 rows); every wave covers all of them
constexpr int kBNW = 4;                  // n-tiles per wave (64 columns); 3 for some shapes (BGemmArgs::nw)
constexpr int kBN = kBWaves * kBNW;      // n-tiles per work-group (256 columns)
constexpr int kMaxSeq = 64;              // sequences in one batched call
constexpr int kBKeys = 512;              // keys (context and block) per batched attention work item
constexpr int kBSplitMax = 8;            // K parts of one batched GEMM output tile
constexpr long kBPartFloats = (long)kBWaves * kBM * kBNW * 256;  // one work-group's partial tile
constexpr int kBCounters = 4096;         // split-K arrival counters (output tiles of one launch)

enum BEpi { BEPI_QKV = 0, BEPI_RESID = 1, BEPI_SWIGLU = 2, BEPI_ARGMAX = 3, BEPI_BIAS16 = 4 };

// Rows of one batched call, passed by value: call sequence i (cache slot seq[i], context
// length L[i]) owns rows off[i] .. off[i+1]-1 of the call's activations; its attention work
// items are ipfx[i] .. ipfx[i+1]-1 (n_kv per range of kBKeys keys of its L + B keys).
struct BRows {
  int n_seq;
  int seq[kMaxSeq];
  int L[kMaxSeq];
  int off[kMaxSeq + 1];
  int ipfx[kMaxSeq + 1];
};

// Y = A W^T with a fused epilogue.  A: fp16 A fragments [layers][Mt][Kt][64 lanes x 16 B]
// (the MFMA A-operand layout of the activations, one plane); W: packed weight tiles in
// fp16 [layers][Nt][Kt][64].  Work-group = (layer, K part,
// 256-column n-group, 128-row m-group); with kg > 1 the K parts of a tile leave fp32
// partial tiles and the last to arrive sums them in K order and runs the epilogue.
struct BGemmArgs {
  const u32x4* A;
  long a_layer;   // u32x4 units between layers
  const u32x4* W;
  long w_layer;
  int Nt, Kt, Mt, M, kg, layers;
  int nw;              // n-tiles per wave: kBNW, or 3 where that fills the CUs better
  const u32x4* zero;   // one zero fragment
  float* part;         // partial tiles [tiles][kg][kBPartFloats]
  unsigned* cnt;       // arrival counters [tiles], 32 words apart, zero between launches
  // QKV (block rows) and KVT (appended context rows): queries [Mt * 16, q_dim] fp32; keys and
  // values (fp16) to the rows' sequence caches at their slots; RoPE at the slot position
  float* Q;
  int q_dim;
  uint16_t* kc;
  uint16_t* vt;
  long seq_stride, cache_layer;
  int layer0, Lcap, hd, q_tiles, kv_tiles;
  const float2* rope;
  // QKV with q_tiles = 0 (context K/V): optional fp32 bias [layers][K kv | V kv], added
  // before the rotation.  BIAS16: optional fp32 bias per output column.
  const float* bias;
  // RESID: residual stream X [M, H] += Y
  float* X;
  int H;
  // SWIGLU: fp16 A fragments of the MLP hidden rows [Mt][out_kt][64]; BIAS16: fp16 A
  // fragments of Y + bias in the same layout
  u32x4* out16;
  int out_kt;
  // ARGMAX: optional logits [M, V]; best (score, id) per (n-group, row); the score is the
  // logit, or with inv_temp > 0 the logit * inv_temp plus the Gumbel noise of draw `draw`
  // under `seed` at the row's (sequence slot, block position)
  float* logits;
  int V;
  float* pmax;
  int* pidx;
  int pld;
  float inv_temp;
  unsigned draw;
  unsigned long long seed;
};

struct BAttnArgs {
  const float* Q;  // [M, n_q * hd], block rows of call sequence i at off[i]
  const uint16_t* kc;
  const uint16_t* vt;
  long seq_stride, cache_layer;
  int layer, Lcap, B, n_q, n_kv, Rpad;
  float qscale;
  float* OP;    // partial outputs [items][Rpad][hd]
  float2* ML;   // [items][Rpad] (max, sum), log2 domain
};

int bgemm_groups(int Nt, int Mt, int nw = kBNW);  // output tiles of one layer
// n 16-byte slots of packed bf16 weight tiles -> fp16 (same layout)
void launch_tiles_to_f16(hipStream_t s, u32x4* dst, const u32x4* src, long n);
void launch_bgemm(hipStream_t s, int epi, const BGemmArgs& g, const BRows& rows);
void launch_bargmax(hipStream_t s, const float* pmax, const int* pidx, int ngroups, int pld, int M, int* tokens);
// RMSNorm of rows of X (or of embedding rows) into fp16 A fragments
void launch_bnorm(hipStream_t s, const float* X, int M, int H, const float* gain, float eps, u32x4* A, int a_kt);
void launch_bembed_norm(hipStream_t s, const uint16_t* embed, const int32_t* ids, int M, int H, int V,
                        const float* gain, float eps, float* X, u32x4* A, int a_kt);
// layer fusion (Eq. 3) of N appended rows for every draft layer, normalised, into fp16 A
// fragments [D][mt_max][H/32][64]
// (hidden: [S, ld, H], rows 0 .. N-1 of each target layer used)
void launch_bfuse(hipStream_t s, const uint16_t* hidden, int N, int ld, int S, int H, int D, const float* alpha,
                  const float* gain, float eps, u32x4* A, int mt_max);
void launch_bfrag_rows(hipStream_t s, const u32x4* A, int n, int H, int D, int mt_max, float* out);
// target rows [S, ld, H] (bf16), rows 0 .. N-1 -> fp16 A fragments of the rows [h^(1); ...; h^(S)] of each
// position, [mt][S*H/32][64] (the input of the DFlash FC layer, Eq. 1)
void launch_bfrag_cat(hipStream_t s, const uint16_t* hidden, int N, int ld, int S, int H, u32x4* A);
void launch_battn(hipStream_t s, int hd, const BAttnArgs& a, const BRows& rows, int items);
void launch_bcomb(hipStream_t s, int hd, const BAttnArgs& a, const BRows& rows, u32x4* out16, int a_kt);

}  // namespace dflare
