// Declarations of the batched draft step (batched.hip): many sequences, each with its own
// context cache, drafted together so that every projection is a GEMM over all their
// block rows.
#pragma once

#include "dflare_impl.h"

namespace dflare {

constexpr int kBM = 8;        // 16-row m-tiles per GEMM work-group (128 rows)
constexpr int kBN = 8;        // 16-column n-tiles per GEMM work-group (128 columns)
constexpr int kMaxSeq = 64;   // sequences in one batched call

enum BEpi { BEPI_QKV = 0, BEPI_RESID = 1, BEPI_SWIGLU = 2 };

// Rows of one batched call, passed by value: call sequence i (cache slot seq[i], context
// length L[i]) owns rows off[i] .. off[i+1]-1 of the call's activations; its attention work
// items are ipfx[i] .. ipfx[i+1]-1 (n_kv per 128-key chunk of its context).
struct BRows {
  int n_seq;
  int seq[kMaxSeq];
  int L[kMaxSeq];
  int off[kMaxSeq + 1];
  int ipfx[kMaxSeq + 1];
};

// Y = A W^T.  A: hi/lo bf16 A fragments [Mt][a_kt][64]; W: packed tiles [Nt][Kt][64].
// Grid: n-groups of kBN tiles x m-groups of kBM tiles x kg K parts, as one dimension.
struct BGemmArgs {
  const u32x4* Ahi;
  const u32x4* Alo;
  int a_kt;
  const u32x4* W;
  int Nt, Kt;
  const u32x4* zero;  // one zero fragment (64 lanes x 16 bytes)
  int Mt, M, kg;
  // plain output: fp32 slices Y[kg][Mt * 16][ldy]
  float* Y;
  int ldy;
  // LM head: row scale, optional logits [M, V], best (logit, id) per (n-group, row)
  const float* rstd;
  float* logits;
  int V;
  float* pmax;
  int* pidx;
  int pld;
};

// Epilogue of a GEMM: sums the kg slices in order, then per operator (see BEpi).
struct BEpiArgs {
  const float* Y;
  int kg, Mpad, ldy;
  int M, N, H;
  const float* rstd;  // row scale (QKV, SWIGLU)
  // RESID: residual stream [M, H] += Y; sums of squares [M][H/16] of the new rows
  float* X;
  float* stats;
  const float* gain;  // gain of the next RMSNorm (RESID)
  // A fragments written (RESID: x * gain, SWIGLU: the MLP hidden rows)
  u32x4* ahi;
  u32x4* alo;
  int a_kt;
  // QKV: rotated queries [M, q_dim]; keys and values to the rows' caches
  float* Q;
  int q_dim;
  uint16_t* kc;
  uint16_t* vt;
  long seq_stride, cache_layer;
  int layer, Lcap, hd, q_tiles, kv_tiles;
  const float2* rope;
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

void launch_bgemm(hipStream_t s, const BGemmArgs& g, bool argmax);
int bgemm_groups(int Nt, int Mt);  // work-groups of one K part
void launch_bargmax(hipStream_t s, const float* pmax, const int* pidx, int ngroups, int pld, int M, int* tokens);
void launch_brstd(hipStream_t s, const float* stats, int n_st, int M, float inv_dim, float eps, float* rstd);
void launch_bembed(hipStream_t s, const uint16_t* embed, const int32_t* ids, int M, int H, int V,
                   const float* gain, float* X, float* stats, u32x4* ahi, u32x4* alo, int a_kt);
void launch_bepi(hipStream_t s, int kind, const BEpiArgs& e, const BRows& rows);
void launch_battn(hipStream_t s, int hd, const BAttnArgs& a, const BRows& rows, int items);
void launch_bcomb(hipStream_t s, int hd, const BAttnArgs& a, const BRows& rows, u32x4* ohi, u32x4* olo, int a_kt);

}  // namespace dflare
