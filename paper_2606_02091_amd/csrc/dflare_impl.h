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

// Epilogue selected by the GEMM template.
enum Epi {
  EPI_RESID = 0,   // out[row, col] += y; per-16-column sums of squares of the result
  EPI_SWIGLU = 1,  // out[row, f] = silu(gate_f) * up_f
  EPI_QKV = 2,     // block Q (RoPE, fp32), block K (RoPE) and V into cache slots L + row
  EPI_KVT = 3,     // context K (RoPE) and V of appended rows into cache slots L + row
  EPI_ARGMAX = 4   // vocabulary-parallel argmax: best (logit, id) of the block per row
};

struct StepParams {  // device-resident, rewritten by a prologue kernel each call
  int L;             // context length before this call
  int n_new;         // rows appended by this call (fuse_append)
  int pos[16];       // block positions (draft_block)
};

struct EpiArgs {
  const StepParams* params;
  float* out;             // RESID: X [M, ldo]; SWIGLU: H [M, ldo]; QKV: Q [B, ldo]
  int ldo;
  float* stats_out;       // RESID: [M, n_stat_out]
  int n_stat_out;
  uint16_t* kc;           // K cache of the layer (QKV) or of layer 0 (KVT): [n_kv, Lcap, hd]
  uint16_t* vt;           // V cache, transposed: [n_kv, hd, Lcap]
  long plane;             // elements from the hi plane of a cache to its lo plane
  long cache_layer_stride;  // elements between consecutive layers' caches (KVT)
  int Lcap;
  int hd;
  int q_tiles;            // QKV: number of Q tiles; KVT: 0
  int kv_tiles;           // tiles of the K region (== tiles of the V region)
  const float2* rope;     // [positions, hd/2] (cos, sin)
  int B;                  // block rows (QKV / ARGMAX)
  // ARGMAX
  int vocab;
  float* pmax;            // [16, blocks]: best logit of each block per row
  int* pidx;              // [16, blocks]: its token id
  float* logits;          // optional debug [B, vocab]
  // RESID / SWIGLU: A fragments of the next GEMM's input (RESID: x * next_gain)
  uint32_t* na_hi;
  uint32_t* na_lo;
  int na_Kt;
  const float* next_gain;
};

struct GemmArgs {
  const u32x4* W;          // packed tiles of layer 0
  long w_layer_stride;     // in u32x4 units (layer = blockIdx.y)
  int Nt, Kt;              // output tiles (16 wide), k tiles (32 deep)
  const u32x4* zero;       // one zero tile (64 x 16 bytes)
  const u32x4* Ahi;        // activation A fragments (hi / lo planes) of layer 0, [m-tiles, Kt, 64]
  const u32x4* Alo;
  long a_layer_stride;     // in u32x4 units
  int M;                   // rows (ignored for KVT, which reads n_new)
  const float* stats;      // optional: per-row partial sums of squares [M, n_stat]; when set the
  long stats_layer_stride; // output rows are scaled by 1/sqrt(sum * inv_dim + eps) (RMSNorm)
  int n_stat;
  float inv_dim, eps;
  EpiArgs e;
};

struct AttnArgs {
  const StepParams* params;
  const float* Q;          // [B, q_dim] fp32, rotated
  const uint16_t* kc;      // [n_kv, Lcap, hd] of the layer (hi plane; lo plane at +plane)
  const uint16_t* vt;      // [n_kv, hd, Lcap]
  long plane;
  int B, n_q, n_kv, q_dim, Lcap, Rpad;
  float qscale;            // log2(e) / sqrt(hd)
  float* opart;            // [chunks, n_kv, Rpad, hd]
  float2* ml;              // [chunks, n_kv, Rpad]
  u32x4* oa_hi;            // combine: A fragments of O [B, q_dim] for the output projection
  u32x4* oa_lo;
  int oa_Kt;
};

// ---- launchers (kernels.hip) ----
void launch_pack(hipStream_t s, u32x4* dst, const uint16_t* src0, const uint16_t* src1,
                 int n_src_rows, int K, int nt_begin, int nt_count, int Kt_total, int mode, int hd);
void launch_bf16_to_f32(hipStream_t s, float* dst, const uint16_t* src, long n);
void launch_prologue(hipStream_t s, StepParams* p, const StepParams& host, const int* ids_src,
                     int* ids_dst, int B);
void launch_embed(hipStream_t s, const uint16_t* embed, const int* ids, int vocab, int H, int B,
                  float* X, float* stats, const float* gain, u32x4* a_hi, u32x4* a_lo);
void launch_fuse(hipStream_t s, const uint16_t* hidden, int n, int S, int H, int D, const float* alpha,
                 const float* gain, float* ustats, u32x4* ua_hi, u32x4* ua_lo, int n_max, int mt_max,
                 StepParams* params, int L);
void launch_fused_rows(hipStream_t s, const u32x4* ua_hi, const u32x4* ua_lo, const float* ustats, int n,
                       int H, int D, int n_max, int mt_max, float eps, float* out);
void launch_gemm(hipStream_t s, int epi, int nt_per_block, int waves, const GemmArgs& a, int layers, int mtiles);
bool gemm_shape_supported(int nt_per_block, int waves);
void launch_argmax_combine(hipStream_t s, const float* pmax, const int* pidx, int groups, int B, int* tokens);
void launch_attention(hipStream_t s, const AttnArgs& a, int hd, int chunk, int n_chunks);
void launch_attn_combine(hipStream_t s, const AttnArgs& a, int hd, int chunk, int n_chunks);

}  // namespace dflare
