// Training-side kernels of the block diffusion draft model and their C-ABI entry points:
//   * anchor attention (Sec. 3.3): the sampled blocks of a sequence are processed together;
//     the rows of block i (anchored at position a_i) attend to the context features of the
//     positions before a_i and to the B positions of their own block, never to another
//     block.  Forward (outputs, log-sum-exp) and backward (dQ, context dK/dV, block dK/dV).
//   * progressive position-weighted cross-entropy (Sec. 4.3, Eq. 5): weights
//     w_k = exp(-(k - 1) / gamma) on the k-th masked position of each block, the loss is
//     their weighted mean; forward and the gradient of the logits.
//
// Matrix products run on v_mfma_f32_16x16x32_bf16 with every operand read straight from
// memory in its operand layout: scores are formed transposed (S^T = K Q^T) where the
// probabilities feed a product over keys (P V, dS K), and untransposed (S = Q K^T) where they
// feed a product over query rows (P^T dO, dS^T Q).  The operands that need the other
// orientation (V^T, K^T, Q^T, dO^T) are written once per call into the workspace by
// transposing kernels; two 16-key (or 16-row) result tiles of a lane hold keys 4q..4q+3 and
// 16+4q..16+4q+3, so the matching operand is read as two 8-byte pieces.
#include <hip/hip_runtime.h>
#include <math.h>

#include <algorithm>
#include <mutex>
#include <type_traits>

#include "device_common.h"
#include "dflare.h"

namespace dflare {

namespace {

constexpr int kTrT = 256;  // threads per work-group (4 waves)
constexpr int kChunkBlocks = 64;  // blocks per partial of the context-key gradients
constexpr int kMaxBlockKeys = 16;  // block size B the training entry points accept

struct AttnShapeT {
  int n_blocks, B, T, n_q, n_kv, hd;
  int G, R, Rp, Tp, Mp;  // heads per group, rows per (block, group), padded rows / context keys / block keys
};

struct AttnT {
  AttnShapeT s;
  const uint16_t *q, *kc, *vc, *kb, *vb;  // bf16 inputs
  const int32_t* anchors;
  // workspace (bf16 transposed copies, fp32 partials)
  uint16_t *kct, *vct, *kbt, *vbt;  // [n_kv][hd][Tp] / [n_kv][hd][n_blocks * 32]
  uint16_t *qt, *dot, *dob;         // [n_kv][n_blocks][hd][Rp] x2, [M][n_q][hd]
  uint16_t *qr, *dor;               // [n_kv][n_blocks][Rp][hd] x2 (rows of a (block, group))
  float2* st;                       // [n_kv][n_blocks][Rp] (lse * log2 e, rowsum(dO O)); (+inf, 0) past R
  float* dsum;                      // [M][n_q] rowsum(dO * O)
  float* part;                      // [nch][T][n_kv][hd] x2 (dK, dV)
  int* order;                       // [n_blocks] blocks by decreasing anchor (work order)
  int nch;
  // outputs
  float *out, *lse;
  const float* dout;
  float *dq, *dkc, *dvc, *dkb, *dvb;
  float scale;
};

__device__ __forceinline__ u32x4 ld16(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }
// keys (or rows) 4q..4q+3 and 16+4q..16+4q+3 of a 32-wide range starting at p
__device__ __forceinline__ u32x4 ld_pair(const uint16_t* p) {
  const u32x2 a = *reinterpret_cast<const u32x2*>(p);
  const u32x2 b = *reinterpret_cast<const u32x2*>(p + 16);
  return u32x4{a[0], a[1], b[0], b[1]};
}
// two fp32 values -> two bf16 (round to nearest even) in one word, by the packed conversion
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t cvt_bf2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{lo, hi}), bf16x2_t));
}
// two result tiles of a lane (4 + 4 values) as one bf16 operand (k order 0..3, then 16..19)
__device__ __forceinline__ u32x4 pack_bf8(f32x4 x, f32x4 y) {
  return u32x4{cvt_bf2(x[0], x[1]), cvt_bf2(x[2], x[3]), cvt_bf2(y[0], y[1]), cvt_bf2(y[2], y[3])};
}
// 2^x by the hardware instruction: results below 2^-126 (far below a bf16 probability's
// resolution) are not kept as denormals; 2^-inf = 0
__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }
// LDS swizzles.  Row tiles (PK 16-byte pieces per row): piece c of row k sits in slot
// c ^ rsw(k), so that one piece of 16 consecutive rows covers all 64 banks.  Transposed tiles
// (4 pieces of 8 keys per dim row d): piece c in slot c ^ tsw(d), the same for 16 dim rows.
template <int PK>
__device__ __forceinline__ int rsw(int k) {
  return PK == 16 ? (k & 15) : ((k >> 1) & 7);
}
__device__ __forceinline__ int tsw(int d) { return (d >> 2) & 3; }

// ---- layout helpers ------------------------------------------------------------------
// src [rows][n_kv][hd] (bf16) -> dst [n_kv][hd][ld], zeros for rows >= nrows; block
// (32-row tile, 32-column tile of n_kv*hd) through a padded LDS tile.
__global__ __launch_bounds__(256) void k_tr_kv_t(const uint16_t* src, int nrows, int cols, int ld, uint16_t* dst) {
  __shared__ uint16_t tile[32][34];
  const int r0 = blockIdx.x * 32, c0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
  for (int y = ty; y < 32; y += 8) {
    const int r = r0 + y, c = c0 + tx;
    tile[y][tx] = (r < nrows && c < cols) ? src[(long)r * cols + c] : (uint16_t)0;
  }
  __syncthreads();
  for (int y = ty; y < 32; y += 8) {
    const int c = c0 + y, r = r0 + tx;
    if (c < cols && r < ld) dst[(long)c * ld + r] = tile[tx][y];
  }
}

// block keys src [n_blocks*B][n_kv][hd] -> dst [n_kv][hd][n_blocks*32]: block i's keys at
// i*32 + j (j < B), zeros for j >= B, so that every 16-byte piece of a block is aligned.
// Work-group = (block i, 256 columns): rows read along the columns into an LDS tile, then each
// column's 32 keys written as four 16-byte pieces.
__global__ __launch_bounds__(256) void k_tr_blk_t(const uint16_t* src, int n_blocks, int B, int cols, uint16_t* dst) {
  __shared__ uint16_t tl[256][kMaxBlockKeys + 2];
  const int i = blockIdx.x, c0 = blockIdx.y * 256, t = threadIdx.x;
  const long ld = (long)n_blocks * 32;
  for (int j = 0; j < B; ++j) tl[t][j] = c0 + t < cols ? src[((long)i * B + j) * cols + c0 + t] : (uint16_t)0;
  __syncthreads();
  for (int e = t; e < 256 * 4; e += 256) {
    const int c = e / 4, pc = e % 4;  // column c0 + c, keys 8 pc .. 8 pc + 7
    if (c0 + c >= cols) continue;
    uint32_t w[4];
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const int j = 8 * pc + 2 * h;
      const uint32_t lo = j < B ? tl[c][j] : 0u, hi = j + 1 < B ? tl[c][j + 1] : 0u;
      w[h] = lo | (hi << 16);
    }
    *reinterpret_cast<u32x4*>(dst + (long)(c0 + c) * ld + (long)i * 32 + 8 * pc) = u32x4{w[0], w[1], w[2], w[3]};
  }
}

// ---- backward operands of (block i, KV head g), one work-group each.  Row r < R of the pair
// is block position r % B of query head g G + r / B; a row is read once (Q, dO, O: HD / 4
// threads, four dims each) and gives dO in bf16 (dob, the input layout), D = rowsum(dO O)
// (dsum), the grouped row copies qr and dor, the pair (lse log2 e, D) (st), and, through an
// LDS tile, the transposed copies qt and dot.  Rows R .. Rp-1 are zeros (st: (+inf, 0)).  The
// LDS tiles [2][HD][Rp] keep each 32-row group with its rows permuted per dim row (r ^ (2
// (d / 4) mod 32)), so that the row-wise writes spread over the banks. ----
template <int HD>
__global__ __launch_bounds__(256) void k_bwd_prep(const uint16_t* q, const float* dout, const float* out,
                                                   const float* lse, AttnShapeT s, uint16_t* dob, float* dsum,
                                                   uint16_t* qr, uint16_t* dor, float2* st, uint16_t* qt,
                                                   uint16_t* dot) {
  extern __shared__ uint16_t tl[];
  constexpr int TPR = HD / 4, RPS = 256 / TPR;
  const int i = blockIdx.x, g = blockIdx.y;
  const int c4 = threadIdx.x % TPR, rs = threadIdx.x / TPR;
  const int d0 = 4 * c4;
  const int swz = (2 * c4) & 31;
  const long tile = (long)g * s.n_blocks + i;
  uint16_t* tlq = tl;
  uint16_t* tld = tl + HD * s.Rp;
  for (int r = rs; r < s.Rp; r += RPS) {
    const bool rv = r < s.R;
    const long rh = rv ? (long)(i * s.B + r % s.B) * s.n_q + g * s.G + r / s.B : 0;
    f32x4 x = zero4(), o = zero4();
    u32x2 qv = {0u, 0u};
    if (rv) {
      x = *reinterpret_cast<const f32x4*>(dout + rh * HD + d0);
      o = *reinterpret_cast<const f32x4*>(out + rh * HD + d0);
      qv = *reinterpret_cast<const u32x2*>(q + rh * HD + d0);
    }
    float acc = (x[0] * o[0] + x[1] * o[1]) + (x[2] * o[2] + x[3] * o[3]);
#pragma unroll
    for (int off = TPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    const u32x2 dv = {f2bf(x[0]) | (f2bf(x[1]) << 16), f2bf(x[2]) | (f2bf(x[3]) << 16)};
    if (rv) *reinterpret_cast<u32x2*>(dob + rh * HD + d0) = dv;
    *reinterpret_cast<u32x2*>(qr + (tile * s.Rp + r) * HD + d0) = qv;
    *reinterpret_cast<u32x2*>(dor + (tile * s.Rp + r) * HD + d0) = dv;
    const int rr = (r & ~31) | ((r & 31) ^ swz);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      tlq[(d0 + e) * s.Rp + rr] = (uint16_t)(qv[e >> 1] >> (16 * (e & 1)));
      tld[(d0 + e) * s.Rp + rr] = (uint16_t)(dv[e >> 1] >> (16 * (e & 1)));
    }
    if (c4 == 0) {
      if (rv) dsum[rh] = acc;
      st[tile * s.Rp + r] = rv ? make_float2(lse[rh] * 1.4426950408889634f, acc) : make_float2(INFINITY, 0.f);
    }
  }
  __syncthreads();
  // transposed copies [g][i][d][Rp]: rows r, r + 1 of dim row d per 4-byte store
  const int half = s.Rp / 2;
  for (int e = threadIdx.x; e < HD * half; e += 256) {
    const int d = e / half, r = 2 * (e % half);
    const int rr = (r & ~31) | ((r & 31) ^ ((2 * (d >> 2)) & 31));
    const long dst = (tile * HD + d) * s.Rp + r;
    *reinterpret_cast<uint32_t*>(qt + dst) = *reinterpret_cast<const uint32_t*>(tlq + d * s.Rp + rr);
    *reinterpret_cast<uint32_t*>(dot + dst) = *reinterpret_cast<const uint32_t*>(tld + d * s.Rp + rr);
  }
}

// ---- work order of the row kernels: the blocks by decreasing anchor (ties by index), so that
// the work-groups with the longest contexts start first and the short ones fill the tail.
// Thread i counts the blocks that go before block i. ----
__global__ __launch_bounds__(256) void k_anchor_order(const int32_t* __restrict__ anchors, int n, int T,
                                                      int* __restrict__ order) {
  __shared__ int part[4][64];
  // lane l of wave q: block i = 64 * blockIdx.x + l against the q-th quarter of the blocks; the
  // quarter's anchors are the same for the whole wave (scalar loads)
  const int l = threadIdx.x & 63, q = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int i = blockIdx.x * 64 + l;
  const int ai = i < n ? min(max(anchors[i], 0), T) : 0;
  const int per = (n + 3) / 4, jb = q * per, je = min(n, jb + per);
  int rank = 0;
#pragma unroll 8
  for (int j = jb; j < je; ++j) {
    const int aj = min(max(anchors[j], 0), T);
    rank += (aj > ai || (aj == ai && j < i)) ? 1 : 0;
  }
  part[q][l] = rank;
  __syncthreads();
  if (q == 0 && i < n) order[part[0][l] + part[1][l] + part[2][l] + part[3][l]] = i;
}

// ---- forward and dQ: work-group (block i, KV head g), blocks taken in the order above; its 4 waves take the 16-row query
// tiles w, w + 4 (TPW tiles each).  Key tiles of 32 (the context before the anchor, then the
// block's own keys) are shared through LDS, double-buffered: LDS-direct loads fill the next
// tile while the current one goes through the matrix cores.  Per stage: K rows (and for dQ
// V rows), 16-byte pieces of key k in slot k*(HD/8) + (c ^ rsw(k)); and the transposed tile
// (V^T, or K^T for dQ), piece c (8 keys) of dim row d in slot d*4 + (c ^ tsw(d)).  Keys a
// block does not see are read from a visible row and masked in the scores.
template <int HD, bool DQ, int TPW>
__global__ __launch_bounds__(kTrT) void k_aatt_rows(AttnT a) {
  constexpr int PK = HD / 8;                   // 16-byte pieces of a key row
  constexpr int KP = 32 * PK, TP = HD * 4;     // pieces of a key-row tile / of a transposed tile
  constexpr int NP = (DQ ? 2 * KP : KP) + TP;  // pieces per stage
  static_assert(NP % 64 == 0, "whole wave loads");
  __shared__ u32x4 lds[2][NP];
  const AttnShapeT& s = a.s;
  const int i = a.order[blockIdx.x], g = blockIdx.y;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int col = lane & 15, q4 = lane >> 4;
  const int QT = (s.R + 15) / 16;
  const int anchor = min(max(a.anchors[i], 0), s.T);
  const int nct = (anchor + 31) / 32;
  const float sl2 = a.scale * 1.4426950408889634f;
  const u32x4 z4 = {0u, 0u, 0u, 0u};
  const uint16_t* tsrc_c = DQ ? a.kct : a.vct;
  const uint16_t* tsrc_b = DQ ? a.kbt : a.vbt;

  // LDS-direct loads of key tile kt into buffer bi.  Each region (K rows, V rows for dQ, the
  // transposed tile) is RW wave-loads; wave w issues loads w, w + 4, ... of each, from a
  // per-tile base plus a per-lane offset fixed for the whole kernel.  Keys past T (the last
  // context tile) and block keys past B read row 0; their scores are masked.
  constexpr int RW = HD / 16, PW = RW / 4;
  int kk[PW], cofs[PW], rofs_b[PW], tofs_c[PW], tofs_b[PW];
#pragma unroll
  for (int t = 0; t < PW; ++t) {
    const int sl = (w + 4 * t) * 64 + lane;
    const int k = sl / PK, d = sl / 4;
    kk[t] = k;
    cofs[t] = ((sl % PK) ^ rsw<PK>(k)) * 8;
    rofs_b[t] = (k < s.B ? k : 0) * s.n_kv * HD + cofs[t];
    const int ct = ((sl % 4) ^ tsw(d)) * 8;
    tofs_c[t] = d * s.Tp + ct;
    tofs_b[t] = d * s.Mp + ct;
  }
  // (source pointers through locals: an array element inside the builtin's argument left the
  // host-side launch stub undefined)
  auto issue = [&](int bi, int t, const uint16_t* sk, const uint16_t* sv, const uint16_t* stt) {
    const int ins = w + 4 * t;
    __builtin_amdgcn_global_load_lds(sk, (LDSP char*)(char*)&lds[bi][ins * 64], 16, 0, 0);
    if constexpr (DQ) __builtin_amdgcn_global_load_lds(sv, (LDSP char*)(char*)&lds[bi][(RW + ins) * 64], 16, 0, 0);
    __builtin_amdgcn_global_load_lds(stt, (LDSP char*)(char*)&lds[bi][((DQ ? 2 : 1) * RW + ins) * 64], 16, 0, 0);
  };
  auto stage = [&](int kt, int bi) {
    if (kt == nct) {  // the block's own keys
      const long r0 = ((long)i * s.B * s.n_kv + g) * HD;
      const uint16_t* bt = tsrc_b + (long)g * HD * s.Mp + (long)i * 32;
#pragma unroll
      for (int t = 0; t < PW; ++t) {
        const int ro = rofs_b[t], to = tofs_b[t];
        issue(bi, t, a.kb + r0 + ro, a.vb + r0 + ro, bt + to);
      }
    } else {
      const long r0 = ((long)kt * 32 * s.n_kv + g) * HD;
      const uint16_t* bt = tsrc_c + (long)g * HD * s.Tp + (long)kt * 32;
      const bool tail = (kt + 1) * 32 > s.T;
#pragma unroll
      for (int t = 0; t < PW; ++t) {
        long ro = r0 + (long)kk[t] * s.n_kv * HD + cofs[t];
        if (tail && kt * 32 + kk[t] >= s.T) ro = (long)g * HD + cofs[t];  // key 0
        const int to = tofs_c[t];
        issue(bi, t, a.kc + ro, a.vc + ro, bt + to);
      }
    }
  };

  // per query tile of this wave: Q (and dO) fragments, softmax state, accumulators
  u32x4 qf[TPW][HD / 32], df[TPW][HD / 32];
  float m[TPW], l[TPW], lse2[TPW], dr[TPW];
  f32x4 o[TPW][HD / 16];
#pragma unroll
  for (int tt = 0; tt < TPW; ++tt) {
    const int r = 16 * (w + 4 * tt) + col;
    const bool rv = r < s.R;
    const int h = g * s.G + (rv ? r / s.B : 0), b = rv ? r % s.B : 0;
    const long qrow = ((long)(i * s.B + b) * s.n_q + h) * HD;
#pragma unroll
    for (int ks = 0; ks < HD / 32; ++ks) {
      qf[tt][ks] = rv ? ld16(a.q + qrow + ks * 32 + 8 * q4) : z4;
      if constexpr (DQ) df[tt][ks] = rv ? ld16(a.dob + qrow + ks * 32 + 8 * q4) : z4;
    }
    m[tt] = -1e30f;  // finite: 2^(-inf - m) = 0 for masked keys before any visible one
    l[tt] = 0.f;
    lse2[tt] = dr[tt] = 0.f;
    if constexpr (DQ) {
      lse2[tt] = rv ? a.lse[(long)(i * s.B + b) * s.n_q + h] * 1.4426950408889634f : 0.f;
      dr[tt] = rv ? a.dsum[(long)(i * s.B + b) * s.n_q + h] : 0.f;
    }
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) o[tt][dt] = zero4();
  }

  const char* L0 = reinterpret_cast<const char*>(&lds[0][0]);
  stage(0, 0);
  wait_vm();
  __syncthreads();
  // one key tile; the buffer index is a compile-time constant (the loop below runs tiles in
  // pairs), so every LDS read takes its buffer offset as an immediate
  auto tile = [&](int kt, auto BI) {
    constexpr int bi = decltype(BI)::value;
    if (kt < nct) stage(kt + 1, bi ^ 1);
    const bool blk = kt == nct;
    const char* Lb = L0 + bi * NP * 16;
    // A-operand rows of this lane: keys 16 x + col
    u32x4 ka[2][HD / 32], va[2][HD / 32];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int ks = 0; ks < HD / 32; ++ks) {
        const int k = 16 * x + col;
        const int sl = k * PK + ((ks * 4 + q4) ^ rsw<PK>(k));
        ka[x][ks] = *reinterpret_cast<const u32x4*>(Lb + sl * 16);
        if constexpr (DQ) va[x][ks] = *reinterpret_cast<const u32x4*>(Lb + (KP + sl) * 16);
      }
    // every key of the tile visible (all context tiles but the last): no masking
    const bool full = !blk && (kt + 1) * 32 <= anchor;
    // transposed operand pieces of this lane (dims 16 dt + col), read once for all its tiles
    u32x4 tpair[HD / 16];
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) {
      const int d = 16 * dt + col;
      const int base = (DQ ? 2 * KP : KP) + d * 4;
      const int c0 = (q4 >> 1) ^ tsw(d), c1 = (2 + (q4 >> 1)) ^ tsw(d);
      const u32x2 lo = *reinterpret_cast<const u32x2*>(Lb + (base + c0) * 16 + (q4 & 1) * 8);
      const u32x2 hi = *reinterpret_cast<const u32x2*>(Lb + (base + c1) * 16 + (q4 & 1) * 8);
      tpair[dt] = u32x4{lo[0], lo[1], hi[0], hi[1]};
    }
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      if (w + 4 * tt >= QT) continue;
      f32x4 s0 = zero4(), s1 = zero4(), p0 = zero4(), p1 = zero4();
#pragma unroll
      for (int ks = 0; ks < HD / 32; ++ks) {
        s0 = mfma(ka[0][ks], qf[tt][ks], s0);
        s1 = mfma(ka[1][ks], qf[tt][ks], s1);
        if constexpr (DQ) {
          p0 = mfma(va[0][ks], df[tt][ks], p0);  // dP^T
          p1 = mfma(va[1][ks], df[tt][ks], p1);
        }
      }
      // raw scores of this lane (keys 4 q4 + e and 16 + 4 q4 + e), -inf where masked; the
      // log2-domain scale sl2 > 0 goes into each exponent as one fma
      float x0[4], x1[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x0[e] = s0[e];
        x1[e] = s1[e];
      }
      if (!full) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int j0 = 4 * q4 + e, j1 = 16 + 4 * q4 + e;
          if (!(blk ? j0 < s.B : kt * 32 + j0 < anchor)) x0[e] = -INFINITY;
          if (!(blk ? j1 < s.B : kt * 32 + j1 < anchor)) x1[e] = -INFINITY;
        }
      }
      u32x4 pb;
      if constexpr (!DQ) {
        // the running maximum moves only when the tile's maximum exceeds it by more than 8
        // (so unnormalised probabilities stay below 2^8); the rescale of O and l then runs
        // for the whole wave, with factor 1 on rows that did not move
        float tm = fmaxf(fmaxf(x0[0], x1[0]), fmaxf(x0[1], x1[1]));
        tm = fmaxf(tm, fmaxf(fmaxf(x0[2], x1[2]), fmaxf(x0[3], x1[3])));
        tm = fmaxf(tm, __shfl_xor(tm, 16));
        tm = fmaxf(tm, __shfl_xor(tm, 32));
        tm *= sl2;  // max of the log2-domain scores (scaling by sl2 > 0 keeps the maximum)
        const bool grow = tm > m[tt] + 8.f;
        if (__builtin_amdgcn_ballot_w64(grow) != 0) {
          const float mn = grow ? tm : m[tt];
          const float corr = ex2(m[tt] - mn);
          l[tt] *= corr;
#pragma unroll
          for (int dt = 0; dt < HD / 16; ++dt) o[tt][dt] *= corr;
          m[tt] = mn;
        }
        float ps = 0.f;
        f32x4 e0, e1;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          e0[e] = ex2(fmaf(x0[e], sl2, -m[tt]));
          e1[e] = ex2(fmaf(x1[e], sl2, -m[tt]));
          ps += e0[e] + e1[e];
        }
        l[tt] += ps;
        pb = pack_bf8(e0, e1);
      } else {
        f32x4 d0, d1;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          d0[e] = ex2(fmaf(x0[e], sl2, -lse2[tt])) * (p0[e] - dr[tt]);
          d1[e] = ex2(fmaf(x1[e], sl2, -lse2[tt])) * (p1[e] - dr[tt]);
        }
        pb = pack_bf8(d0, d1);
      }
      // O^T += V^T P^T (forward) or dQ^T += K^T dS^T
#pragma unroll
      for (int dt = 0; dt < HD / 16; ++dt) o[tt][dt] = mfma(tpair[dt], pb, o[tt][dt]);
    }
    wait_vm();
    __syncthreads();
  };
  for (int kt = 0; kt <= nct; kt += 2) {
    tile(kt, std::integral_constant<int, 0>{});
    if (kt + 1 <= nct) tile(kt + 1, std::integral_constant<int, 1>{});
  }
#pragma unroll
  for (int tt = 0; tt < TPW; ++tt) {
    const int r = 16 * (w + 4 * tt) + col;
    if (w + 4 * tt >= QT || r >= s.R) continue;
    const int h = g * s.G + r / s.B, b = r % s.B;
    const long qrow = ((long)(i * s.B + b) * s.n_q + h) * HD;
    float out_scale;
    if constexpr (!DQ) {
      float lt = l[tt];
      lt += __shfl_xor(lt, 16);
      lt += __shfl_xor(lt, 32);
      out_scale = 1.f / lt;
      if (q4 == 0) a.lse[(long)(i * s.B + b) * s.n_q + h] = (m[tt] + log2f(lt)) * 0.6931471805599453f;
    } else {
      out_scale = a.scale;
    }
    float* dst = (DQ ? a.dq : a.out) + qrow;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) *reinterpret_cast<f32x4*>(dst + 16 * dt + 4 * q4) = o[tt][dt] * out_scale;
  }
}

// ---- block-key dK, dV: work-group (block ib, KV head g); wave w takes the block's 32-row
// pairs w, w + 4, ... and the 4 waves' sums are added in wave order ----
template <int HD>
__global__ __launch_bounds__(kTrT) void k_aatt_kvb(AttnT a) {
  constexpr int NX = kMaxBlockKeys / 16;  // 16-key tiles of a block's keys (B <= kMaxBlockKeys)
  const AttnShapeT& s = a.s;
  const int g = blockIdx.y;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int col = lane & 15, q4 = lane >> 4;
  const float sl2 = a.scale * 1.4426950408889634f;
  const int NP = s.Rp / 32;  // 32-row pairs of a (block, group)
  const u32x4 z4 = {0u, 0u, 0u, 0u};
  const int ib = blockIdx.x;
  f32x4 dk[HD / 16][NX], dv[HD / 16][NX];
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt)
#pragma unroll
    for (int x = 0; x < NX; ++x) dk[dt][x] = dv[dt][x] = zero4();
  // B-operand rows (keys) of this lane: key 16x + col of the tile
  u32x4 kf[NX][HD / 32], vf[NX][HD / 32];
#pragma unroll
  for (int x = 0; x < NX; ++x) {
    const int j = 16 * x + col;
    const bool ok = j < s.B;
    const long row = ok ? ((long)(ib * s.B + j) * s.n_kv + g) * HD : 0;
    const uint16_t* kp = a.kb + row;
    const uint16_t* vp = a.vb + row;
#pragma unroll
    for (int ks = 0; ks < HD / 32; ++ks) {
      kf[x][ks] = ok ? ld16(kp + ks * 32 + 8 * q4) : z4;
      vf[x][ks] = ok ? ld16(vp + ks * 32 + 8 * q4) : z4;
    }
  }
  const int i = ib;
  for (int pr = w; pr < NP; pr += 4) {
    // S = Q K^T and dP = dO V^T for rows 32 pr + 16 y + (4 q4 + e) (y = 0, 1), keys 16x + col
    f32x4 sc[2][NX], dp[2][NX];
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int x = 0; x < NX; ++x) sc[y][x] = dp[y][x] = zero4();
#pragma unroll
    for (int y = 0; y < 2; ++y) {
      const int r = 32 * pr + 16 * y + col;  // A row of this lane
      const bool rv = r < s.R;
      const long qrow = rv ? ((long)(i * s.B + r % s.B) * s.n_q + g * s.G + r / s.B) * HD : 0;
#pragma unroll
      for (int ks = 0; ks < HD / 32; ++ks) {
        const u32x4 qa = rv ? ld16(a.q + qrow + ks * 32 + 8 * q4) : z4;
        const u32x4 da = rv ? ld16(a.dob + qrow + ks * 32 + 8 * q4) : z4;
#pragma unroll
        for (int x = 0; x < NX; ++x) {
          sc[y][x] = mfma(qa, kf[x][ks], sc[y][x]);
          dp[y][x] = mfma(da, vf[x][ks], dp[y][x]);
        }
      }
    }
    // P and dS at this lane's values: row 32 pr + 16 y + 4 q4 + e, key 16 x + col
    f32x4 P[2][NX], dS[2][NX];
#pragma unroll
    for (int y = 0; y < 2; ++y) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 32 * pr + 16 * y + 4 * q4 + e;
        const bool rv = r < s.R;
        const long rh = rv ? (long)(i * s.B + r % s.B) * s.n_q + g * s.G + r / s.B : 0;
        const float lse2 = rv ? a.lse[rh] * 1.4426950408889634f : 0.f;
        const float dr = rv ? a.dsum[rh] : 0.f;
#pragma unroll
        for (int x = 0; x < NX; ++x) {
          const int j = 16 * x + col;
          const bool ok = rv && j < s.B;
          const float p = ok ? ex2(fmaf(sc[y][x][e], sl2, -lse2)) : 0.f;
          P[y][x][e] = p;
          dS[y][x][e] = p * (dp[y][x][e] - dr);
        }
      }
    }
    // dV^T += dO^T P, dK^T += Q^T dS: A rows = dims d = 16 dt + col, k = the pair's 32 rows
    const long tb = ((long)g * s.n_blocks + i) * HD * s.Rp + 32 * pr + 4 * q4;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) {
      const long off = tb + (long)(16 * dt + col) * s.Rp;
      const u32x4 doa = ld_pair(a.dot + off);
      const u32x4 qa = ld_pair(a.qt + off);
#pragma unroll
      for (int x = 0; x < NX; ++x) {
        dv[dt][x] = mfma(doa, pack_bf8(P[0][x], P[1][x]), dv[dt][x]);
        dk[dt][x] = mfma(qa, pack_bf8(dS[0][x], dS[1][x]), dk[dt][x]);
      }
    }
  }
  // sum the 4 waves' tiles in wave order through LDS, 8 tiles per round
  __shared__ f32x4 red[3][8][64];
  constexpr int NT = HD / 16 * NX * 2;  // tiles per wave (dK, dV)
  static_assert(NT % 8 == 0, "8 tiles per round");
#pragma unroll
  for (int r0 = 0; r0 < NT; r0 += 8) {
    if (w > 0) {
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int tI = r0 + u, kind = tI / (HD / 16 * NX), rem = tI % (HD / 16 * NX);
        red[w - 1][u][lane] = kind == 0 ? dk[rem / NX][rem % NX] : dv[rem / NX][rem % NX];
      }
    }
    __syncthreads();
    if (w == 0) {
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int tI = r0 + u, kind = tI / (HD / 16 * NX), rem = tI % (HD / 16 * NX);
        const int dt = rem / NX, x = rem % NX;
        f32x4 v = kind == 0 ? dk[dt][x] : dv[dt][x];
        v += red[0][u][lane];
        v += red[1][u][lane];
        v += red[2][u][lane];
        if (kind == 0) v *= a.scale;
        // tile (dims 16 dt + 4 q4 + e, key 16 x + col)
        const int j = 16 * x + col;
        if (j < s.B) {
          const long row = (long)(ib * s.B + j);
          float* dst = (kind == 0 ? a.dkb : a.dvb) + (row * s.n_kv + g) * HD + 16 * dt + 4 * q4;
          *reinterpret_cast<f32x4*>(dst) = v;
        }
      }
    }
    __syncthreads();
  }
}

// ---- context dK, dV: work-group (64-key tile kt, KV head g, chunk z of 64 blocks); wave w
// owns keys 64 kt + 16 w + (0..15) (its K and V rows held as operand fragments).  The
// waves walk the chunk's (block, 32-row pair) units together: each unit's Q rows, dO rows,
// Q^T and dO^T tiles (from the grouped copies) go through swizzled LDS, double-buffered with
// LDS-direct loads one unit ahead; per unit a wave forms S = Q K^T and dP = dO V^T for its keys
// and accumulates dV^T += dO^T P and dK^T += Q^T dS.  Writes this chunk's partial dK, dV.
// Work-groups are numbered so that the 8 XCDs (which take work-groups round-robin) each run
// whole (group, chunk) sets, whose units then stay in that XCD's L2. ----
template <int HD>
__global__ __launch_bounds__(kTrT, 2) void k_aatt_kvc(AttnT a) {
  constexpr int PK = HD / 8;                  // 16-byte pieces of a row
  constexpr int RW = HD / 16;                 // wave-loads of one 32-row (or transposed) tile
  constexpr int PW = RW / 4;                  // of them per wave
  constexpr int NPc = 4 * RW * 64;            // Q, dO, Q^T, dO^T
  __shared__ u32x4 lds[2][NPc];
  const AttnShapeT& s = a.s;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int col = lane & 15, q4 = lane >> 4;
  // work-group -> (kt, g, z)
  const int nkt = gridDim.x;
  const int N = nkt * gridDim.y * gridDim.z;
  const int n = blockIdx.x + nkt * (blockIdx.y + gridDim.y * blockIdx.z);
  const int xq = N / 8, xr = N % 8, x8 = n % 8;
  const int lg = x8 * xq + min(x8, xr) + n / 8;
  const int kt = lg % nkt, g = (lg / nkt) % s.n_kv, z = lg / (nkt * s.n_kv);

  const float sl2 = a.scale * 1.4426950408889634f;
  const u32x4 z4 = {0u, 0u, 0u, 0u};
  const int NPr = s.Rp / 32;
  const int i0 = z * kChunkBlocks, i1 = min(s.n_blocks, i0 + kChunkBlocks);
  const int key0 = kt * 64;
  const int myk = key0 + 16 * w + col;
  const bool kok = myk < s.T;
  u32x4 kf[HD / 32], vf[HD / 32];
  {
    const long row = kok ? ((long)myk * s.n_kv + g) * HD : 0;
#pragma unroll
    for (int ks = 0; ks < HD / 32; ++ks) {
      kf[ks] = kok ? ld16(a.kc + row + ks * 32 + 8 * q4) : z4;
      vf[ks] = kok ? ld16(a.vc + row + ks * 32 + 8 * q4) : z4;
    }
  }
  f32x4 dk[HD / 16], dv[HD / 16];
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt) dk[dt] = dv[dt] = zero4();

  // this lane's source offsets of its wave-loads t of a tile (same for every unit): row tiles
  // (32 rows x HD, row-major) and transposed tiles (HD dim rows x Rp)
  int roff[PW], toff[PW];
#pragma unroll
  for (int t = 0; t < PW; ++t) {
    const int sl = (w + 4 * t) * 64 + lane;
    const int rr = sl / PK, d = sl / 4;
    roff[t] = rr * HD + ((sl % PK) ^ rsw<PK>(rr)) * 8;
    toff[t] = d * s.Rp + ((sl % 4) ^ tsw(d)) * 8;
  }
  // the chunk's anchors, one block per lane (a chunk is 64 blocks), and the blocks that see a
  // key of this tile as a bit mask, walked in block order
  static_assert(kChunkBlocks == 64, "one block per lane");
  const int anc = lane < i1 - i0 ? min(max(a.anchors[i0 + lane], 0), s.T) : 0;
  uint64_t left = __builtin_amdgcn_ballot_w64(anc > key0);
  auto take_block = [&]() {
    if (left == 0) return -1;
    const int j = __builtin_ctzll(left);
    left &= left - 1;
    return j;
  };
  auto stage = [&](int j, int pr, int bi) {
    const int i = i0 + j;
    const long tile = (long)g * s.n_blocks + i;
    const uint16_t* rq = a.qr + (tile * s.Rp + 32 * pr) * HD;
    const uint16_t* rd = a.dor + (tile * s.Rp + 32 * pr) * HD;
    const uint16_t* tq = a.qt + tile * HD * s.Rp + 32 * pr;
    const uint16_t* td = a.dot + tile * HD * s.Rp + 32 * pr;
#pragma unroll
    for (int t = 0; t < PW; ++t) {
      const int ins = w + 4 * t;
      // (source pointers through locals: an array element inside the builtin's argument left
      // the host-side launch stub of this kernel undefined)
      const uint16_t* sq = rq + roff[t];
      const uint16_t* sd = rd + roff[t];
      const uint16_t* sqt = tq + toff[t];
      const uint16_t* sdt = td + toff[t];
      __builtin_amdgcn_global_load_lds(sq, (LDSP char*)(char*)&lds[bi][(0 * RW + ins) * 64], 16, 0, 0);
      __builtin_amdgcn_global_load_lds(sd, (LDSP char*)(char*)&lds[bi][(1 * RW + ins) * 64], 16, 0, 0);
      __builtin_amdgcn_global_load_lds(sqt, (LDSP char*)(char*)&lds[bi][(2 * RW + ins) * 64], 16, 0, 0);
      __builtin_amdgcn_global_load_lds(sdt, (LDSP char*)(char*)&lds[bi][(3 * RW + ins) * 64], 16, 0, 0);
    }
  };
  // (lse * log2 e, D) of this lane's result rows 32 pr + 16 y + 4 q4 + (0..3)
  auto row_stats = [&](int j, int pr, f32x4* st4) {
    const int i = i0 + j;
    const float2* p = a.st + ((long)g * s.n_blocks + i) * s.Rp + 32 * pr + 4 * q4;
#pragma unroll
    for (int y = 0; y < 2; ++y) {
      st4[2 * y] = *reinterpret_cast<const f32x4*>(p + 16 * y);
      st4[2 * y + 1] = *reinterpret_cast<const f32x4*>(p + 16 * y + 2);
    }
  };

  const char* L0 = reinterpret_cast<const char*>(&lds[0][0]);
  int cj = take_block(), cp = 0;  // current unit: block i0 + cj, row pair cp
  f32x4 cst[4], nst[4];
  if (cj >= 0) {
    stage(cj, cp, 0);
    row_stats(cj, cp, cst);
  }
  wait_vm();
  __syncthreads();
  // one unit; the buffer index is a compile-time constant (units run in pairs), so every LDS
  // read takes its buffer offset as an immediate
  auto unit = [&](auto BI) {
    constexpr int bi = decltype(BI)::value;
    int nj = cj, np = cp + 1;
    if (np == NPr) {
      np = 0;
      nj = take_block();
    }
    if (nj >= 0) {
      stage(nj, np, bi ^ 1);
      row_stats(nj, np, nst);
    }
    const int anchor = __builtin_amdgcn_readlane(anc, cj);
    const bool vis = myk < anchor;  // this lane's key (column of every result tile)
    const char* Lb = L0 + bi * NPc * 16;
    // S = Q K^T, dP = dO V^T: A rows = pair rows 16 y + col
    f32x4 sc[2], dp[2];
#pragma unroll
    for (int y = 0; y < 2; ++y) {
      sc[y] = dp[y] = zero4();
      const int rr = 16 * y + col;
#pragma unroll
      for (int ks = 0; ks < HD / 32; ++ks) {
        const int sl = rr * PK + ((ks * 4 + q4) ^ rsw<PK>(rr));
        const u32x4 qa = *reinterpret_cast<const u32x4*>(Lb + sl * 16);
        const u32x4 da = *reinterpret_cast<const u32x4*>(Lb + (RW * 64 + sl) * 16);
        sc[y] = mfma(qa, kf[ks], sc[y]);
        dp[y] = mfma(da, vf[ks], dp[y]);
      }
    }
    f32x4 P[2], dS[2];
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const f32x4 sv = cst[2 * y + (e >> 1)];
        const float l2 = sv[2 * (e & 1)], dr = sv[2 * (e & 1) + 1];
        const float p = vis ? ex2(fmaf(sc[y][e], sl2, -l2)) : 0.f;
        P[y][e] = p;
        dS[y][e] = p * (dp[y][e] - dr);
      }
    const u32x4 pb = pack_bf8(P[0], P[1]), sb = pack_bf8(dS[0], dS[1]);
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) {
      const int d = 16 * dt + col;
      const int c0 = (q4 >> 1) ^ tsw(d), c1 = (2 + (q4 >> 1)) ^ tsw(d);
      const int bq = 2 * RW * 64 + d * 4, bd = 3 * RW * 64 + d * 4;
      const u32x2 q0 = *reinterpret_cast<const u32x2*>(Lb + (bq + c0) * 16 + (q4 & 1) * 8);
      const u32x2 q1 = *reinterpret_cast<const u32x2*>(Lb + (bq + c1) * 16 + (q4 & 1) * 8);
      const u32x2 o0 = *reinterpret_cast<const u32x2*>(Lb + (bd + c0) * 16 + (q4 & 1) * 8);
      const u32x2 o1 = *reinterpret_cast<const u32x2*>(Lb + (bd + c1) * 16 + (q4 & 1) * 8);
      dv[dt] = mfma(u32x4{o0[0], o0[1], o1[0], o1[1]}, pb, dv[dt]);
      dk[dt] = mfma(u32x4{q0[0], q0[1], q1[0], q1[1]}, sb, dk[dt]);
    }
    wait_vm();
    __syncthreads();
#pragma unroll
    for (int e = 0; e < 4; ++e) cst[e] = nst[e];
    cj = nj;
    cp = np;
  };
  while (cj >= 0) {
    unit(std::integral_constant<int, 0>{});
    if (cj < 0) break;
    unit(std::integral_constant<int, 1>{});
  }
  if (kok) {
    float* pk = a.part + (((long)z * s.T + myk) * s.n_kv + g) * HD;
    float* pv = a.part + ((((long)a.nch + z) * s.T + myk) * s.n_kv + g) * HD;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) {
      *reinterpret_cast<f32x4*>(pk + 16 * dt + 4 * q4) = dk[dt] * a.scale;
      *reinterpret_cast<f32x4*>(pv + 16 * dt + 4 * q4) = dv[dt];
    }
  }
}

// context dK, dV = the chunks' partials added in chunk order
__global__ void k_aatt_sum(const float* part, int nch, long n, float* dk, float* dv) {
  for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < n; e += (long)gridDim.x * blockDim.x) {
    float sk = 0.f, sv = 0.f;
    for (int c = 0; c < nch; ++c) {
      sk += part[(long)c * n + e];
      sv += part[((long)nch + c) * n + e];
    }
    dk[e] = sk;
    dv[e] = sv;
  }
}

// ---- weighted CE (Eq. 5).  The row weights and 1 / sum w depend on labels and block positions
// only and come first; then each row's log-sum-exp, CE and gradient in one work-group pass over
// the row twice (the second read finds the row in the memory-side cache: gridDim.x rows are in
// flight at a time); last, the loss in row order. ----
constexpr int kCeT = 1024;       // threads of the row work-group
constexpr int kCeRows = 256;     // rows in flight (work-groups)

// w[r] = exp(-(b - 1) / gamma) for block position b = r mod B > 0 with a label in range, else 0;
// 1 / sum w in fp64, summed in the loss kernel's order
__global__ __launch_bounds__(256) void k_wce_weights(const int32_t* labels, int rows, int V, int B, float gamma,
                                                     float* w, float* inv_wsum) {
  __shared__ double sw[256];
  double a = 0.0;
  for (int r = threadIdx.x; r < rows; r += 256) {
    const int b = r % B, y = labels[r];
    const float wr = (b > 0 && y >= 0 && y < V) ? expf(-(float)(b - 1) / gamma) : 0.f;
    w[r] = wr;
    a += wr;
  }
  sw[threadIdx.x] = a;
  __syncthreads();
  for (int k = 128; k > 0; k >>= 1) {
    if ((int)threadIdx.x < k) sw[threadIdx.x] += sw[threadIdx.x + k];
    __syncthreads();
  }
  if (threadIdx.x == 0) inv_wsum[0] = sw[0] > 0.0 ? (float)(1.0 / sw[0]) : 0.f;
}

// per row: lse (log2 domain: max of z log2 e, sum of 2^(z log2 e - max)), ce = lse - z[label]
// for rows that take part, and dz = (w / sum w) (softmax(z) - onehot(label)), four values per
// thread per step where the row allows 16-byte accesses (V % 4 == 0)
__global__ __launch_bounds__(kCeT) void k_wce_fused(const float* logits, const int32_t* labels, int rows, int V,
                                                    int B, const float* w, const float* inv_wsum, float* ce_out,
                                                    float* dz) {
  __shared__ float sm[kCeT / 64], ss[kCeT / 64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const float L2E = 1.4426950408889634f;
  const int V4 = (V % 4 == 0) ? V / 4 : 0;
  const float inv = inv_wsum[0];
  for (int row = blockIdx.x; row < rows; row += gridDim.x) {
    const float* z = logits + (long)row * V;
    float m = -INFINITY, sum = 0.f;
    for (int v = threadIdx.x; v < V4; v += kCeT) {
      const f32x4 x = reinterpret_cast<const f32x4*>(z)[v];
      const float t0 = x[0] * L2E, t1 = x[1] * L2E, t2 = x[2] * L2E, t3 = x[3] * L2E;
      const float m4 = fmaxf(fmaxf(t0, t1), fmaxf(t2, t3));
      if (m4 > m) {
        sum *= ex2(m - m4);
        m = m4;
      }
      sum += (ex2(t0 - m) + ex2(t1 - m)) + (ex2(t2 - m) + ex2(t3 - m));
    }
    for (int v = 4 * V4 + threadIdx.x; v < V; v += kCeT) {
      const float t = z[v] * L2E;
      if (t > m) {
        sum *= ex2(m - t);
        m = t;
      }
      sum += ex2(t - m);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const float om = __shfl_xor(m, off), os = __shfl_xor(sum, off);
      const float nm = fmaxf(m, om);
      sum = (nm == -INFINITY) ? 0.f : sum * ex2(m - nm) + os * ex2(om - nm);
      m = nm;
    }
    if (lane == 0) {
      sm[wv] = m;
      ss[wv] = sum;
    }
    __syncthreads();
    float M = sm[0], S = ss[0];
#pragma unroll
    for (int k = 1; k < kCeT / 64; ++k) {
      const float nm = fmaxf(M, sm[k]);
      S = S * ex2(M - nm) + ss[k] * ex2(sm[k] - nm);
      M = nm;
    }
    __syncthreads();  // sm, ss are rewritten by the next row
    const float lse2 = M + log2f(S);
    const int y = labels[row];
    const bool on = row % B > 0 && y >= 0 && y < V;
    if (threadIdx.x == 0) ce_out[row] = on ? lse2 * 0.6931471805599453f - z[y] : 0.f;
    const float c = w[row] * inv;
    float* d = dz + (long)row * V;
    const int y4 = (on && c != 0.f) ? y >> 2 : -1;
    for (int v = threadIdx.x; v < V4; v += kCeT) {
      f32x4 o = f32x4{0.f, 0.f, 0.f, 0.f};
      if (c != 0.f) {
        const f32x4 x = reinterpret_cast<const f32x4*>(z)[v];
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = c * ex2(fmaf(x[e], L2E, -lse2));
        if (v == y4) o[y & 3] -= c;
      }
      __builtin_nontemporal_store(o, reinterpret_cast<f32x4*>(d) + v);
    }
    for (int v = 4 * V4 + threadIdx.x; v < V; v += kCeT)
      d[v] = c == 0.f ? 0.f : c * ex2(fmaf(z[v], L2E, -lse2)) - (on && v == y ? c : 0.f);
  }
}

// The same per row with the whole row held on chip: one work-group per CU (its LDS share is
// the CU's), kCeOR 16-byte pieces per thread in registers and kCeOL in LDS, so that the row is
// read from memory once; the max, sum and gradient sweeps run over the held values.  Piece v of
// the row: registers slot k of thread t for v = k kCeOT + t, else LDS slot v - kCeOR kCeOT.  For
// rows of kCeOMin .. kCeOCap values (a multiple of 4), so that every register slot is inside the
// row (no per-slot bounds masks to keep).
constexpr int kCeOT = 256;
constexpr int kCeOR = 109;
constexpr int kCeOL = 10224;
constexpr long kCeOCap = ((long)kCeOR * kCeOT + kCeOL) * 4;  // values of a row held on chip
constexpr long kCeOMin = (long)kCeOR * kCeOT * 4;

__global__ __launch_bounds__(kCeOT) void k_wce_chip(const float* logits, const int32_t* labels, int rows, int V,
                                                   int B, const float* w, const float* inv_wsum, float* ce_out,
                                                   float* dz) {
  __shared__ f32x4 lrow[kCeOL];
  __shared__ float red[kCeOT / 64], redm[kCeOT / 64];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const float L2E = 1.4426950408889634f;
  const int V4 = V / 4;
  const float inv = inv_wsum[0];
  for (int row = blockIdx.x; row < rows; row += gridDim.x) {
    const f32x4* z4 = reinterpret_cast<const f32x4*>(logits + (long)row * V);
    f32x4 r[kCeOR];
#pragma unroll
    for (int k = 0; k < kCeOR; ++k) r[k] = z4[k * kCeOT + tid];
    // the rest of the row into LDS (pieces past the row re-read piece 0 and are skipped below)
    for (int m0 = wv * 64; m0 < kCeOL; m0 += kCeOT) {
      const int v = kCeOR * kCeOT + m0 + lane;
      const f32x4* src = z4 + (v < V4 ? v : 0);
      __builtin_amdgcn_global_load_lds(src, (LDSP char*)(char*)&lrow[m0], 16, 0, 0);
    }
    const int nl = min(kCeOL, max(0, V4 - kCeOR * kCeOT));  // LDS pieces of this row
    // running (max, sum) of the log2-domain values, one 16-byte piece at a time (the register
    // pieces in load order, so the sweep follows their arrival), then the LDS pieces
    float m = -INFINITY, sum = 0.f;
    auto take4 = [&](f32x4 x) {
      const float t0 = x[0] * L2E, t1 = x[1] * L2E, t2 = x[2] * L2E, t3 = x[3] * L2E;
      const float m4 = fmaxf(fmaxf(t0, t1), fmaxf(t2, t3));
      if (m4 > m) {
        sum *= ex2(m - m4);
        m = m4;
      }
      sum += (ex2(t0 - m) + ex2(t1 - m)) + (ex2(t2 - m) + ex2(t3 - m));
    };
#pragma unroll
    for (int k = 0; k < kCeOR; ++k) take4(r[k]);
    wait_vm();
    __syncthreads();
    for (int j = tid; j < nl; j += kCeOT) take4(lrow[j]);
    // combine the threads' (max, sum) pairs
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const float om = __shfl_xor(m, off), os = __shfl_xor(sum, off);
      const float nm = fmaxf(m, om);
      sum = (nm == -INFINITY) ? 0.f : sum * ex2(m - nm) + os * ex2(om - nm);
      m = nm;
    }
    if (lane == 0) {
      redm[wv] = m;
      red[wv] = sum;
    }
    __syncthreads();
    float M = redm[0], S = red[0];
#pragma unroll
    for (int k = 1; k < kCeOT / 64; ++k) {
      const float nm = fmaxf(M, redm[k]);
      S = S * ex2(M - nm) + red[k] * ex2(redm[k] - nm);
      M = nm;
    }
    __syncthreads();  // red, redm are rewritten by the next row
    const float lse2 = M + log2f(S);
    const int y = labels[row];
    const bool on = row % B > 0 && y >= 0 && y < V;
    if (tid == 0) ce_out[row] = on ? lse2 * 0.6931471805599453f - logits[(long)row * V + y] : 0.f;
    const float c = w[row] * inv;
    // (c = 0 rows: c p = 0 for every value, so no branch per piece)
    f32x4* d4 = reinterpret_cast<f32x4*>(dz + (long)row * V);
    auto grad = [&](f32x4 x, int v) {
      f32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = c * ex2(fmaf(x[e], L2E, -lse2));
      __builtin_nontemporal_store(o, d4 + v);
    };
#pragma unroll
    for (int k = 0; k < kCeOR; ++k) grad(r[k], k * kCeOT + tid);
    for (int j = tid; j < nl; j += kCeOT) grad(lrow[j], kCeOR * kCeOT + j);
    // the label's value, c p - c, rewritten by the thread that stored its piece (a thread's
    // stores to one address land in program order)
    if (on) {
      const int y4 = y >> 2, rest = y4 - kCeOR * kCeOT;
      if ((rest < 0 ? y4 % kCeOT : rest % kCeOT) == tid) {
        const float zy = logits[(long)row * V + y];
        dz[(long)row * V + y] = c * ex2(fmaf(zy, L2E, -lse2)) - c;
      }
    }
    __syncthreads();  // lrow is refilled by the next row
  }
}

// loss = sum w ce / sum w over the rows, in row order (one work-group)
__global__ __launch_bounds__(256) void k_wce_loss(const float* w, const float* ce, int rows, float* loss) {
  __shared__ double sw[256], sl[256];
  double a = 0.0, c = 0.0;
  for (int r = threadIdx.x; r < rows; r += 256) {
    a += w[r];
    c += (double)w[r] * ce[r];
  }
  sw[threadIdx.x] = a;
  sl[threadIdx.x] = c;
  __syncthreads();
  for (int k = 128; k > 0; k >>= 1) {
    if ((int)threadIdx.x < k) {
      sw[threadIdx.x] += sw[threadIdx.x + k];
      sl[threadIdx.x] += sl[threadIdx.x + k];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    loss[0] = sw[0] > 0.0 ? (float)(sl[0] / sw[0]) : 0.f;
  }
}

}  // namespace

// ---- entry points ----------------------------------------------------------------------

static AttnShapeT att_shape(int n_blocks, int B, int T, int n_q, int n_kv, int hd) {
  AttnShapeT s{};
  s.n_blocks = n_blocks;
  s.B = B;
  s.T = T;
  s.n_q = n_q;
  s.n_kv = n_kv;
  s.hd = hd;
  s.G = n_q / n_kv;
  s.R = s.G * B;
  s.Rp = (s.R + 31) / 32 * 32;
  s.Tp = (T + 31) / 32 * 32 + 32;
  s.Mp = n_blocks * 32;
  return s;
}

static int att_check(int n_blocks, int B, int T, int n_q, int n_kv, int hd) {
  if (n_blocks < 1 || B < 1 || B > kMaxBlockKeys || T < 0 || n_q < 1 || n_kv < 1 || n_q % n_kv) return DFLARE_ERR_INVALID_ARG;
  if (hd != 64 && hd != 128) return DFLARE_ERR_UNSUPPORTED;
  if ((n_q / n_kv) * B > 128) return DFLARE_ERR_UNSUPPORTED;
  return DFLARE_OK;
}

struct WsLayout {
  size_t kct, vct, kbt, vbt, qt, dot, qr, dor, st, dob, dsum, part, order, total;
  int nch;
};

static WsLayout ws_layout(const AttnShapeT& s) {
  WsLayout L{};
  auto al = [](size_t x) { return (x + 255) / 256 * 256; };
  size_t o = 0;
  const size_t ctx_t = (size_t)s.n_kv * s.hd * s.Tp * 2, blk_t = (size_t)s.n_kv * s.hd * s.Mp * 2;
  const size_t grp = (size_t)s.n_kv * s.n_blocks * s.hd * s.Rp * 2;
  const size_t rows = (size_t)s.n_blocks * s.B * s.n_q;
  L.nch = (s.n_blocks + kChunkBlocks - 1) / kChunkBlocks;
  L.kct = o; o = al(o + ctx_t);
  L.vct = o; o = al(o + ctx_t);
  L.kbt = o; o = al(o + blk_t);
  L.vbt = o; o = al(o + blk_t);
  L.qt = o; o = al(o + grp);
  L.dot = o; o = al(o + grp);
  L.qr = o; o = al(o + grp);
  L.dor = o; o = al(o + grp);
  L.st = o; o = al(o + (size_t)s.n_kv * s.n_blocks * s.Rp * 8);
  L.dob = o; o = al(o + rows * s.hd * 2);
  L.dsum = o; o = al(o + rows * 4);
  L.part = o; o = al(o + (size_t)2 * L.nch * s.T * s.n_kv * s.hd * 4);
  L.order = o; o = al(o + (size_t)s.n_blocks * 4);
  L.total = o;
  return L;
}

static AttnT att_args(const AttnShapeT& s, const void* q, const void* kc, const void* vc, const void* kb,
                      const void* vb, const int32_t* anchors, void* ws) {
  const WsLayout L = ws_layout(s);
  char* w = static_cast<char*>(ws);
  AttnT a{};
  a.s = s;
  a.q = (const uint16_t*)q;
  a.kc = (const uint16_t*)kc;
  a.vc = (const uint16_t*)vc;
  a.kb = (const uint16_t*)kb;
  a.vb = (const uint16_t*)vb;
  a.anchors = anchors;
  a.kct = (uint16_t*)(w + L.kct);
  a.vct = (uint16_t*)(w + L.vct);
  a.kbt = (uint16_t*)(w + L.kbt);
  a.vbt = (uint16_t*)(w + L.vbt);
  a.qt = (uint16_t*)(w + L.qt);
  a.dot = (uint16_t*)(w + L.dot);
  a.dob = (uint16_t*)(w + L.dob);
  a.qr = (uint16_t*)(w + L.qr);
  a.dor = (uint16_t*)(w + L.dor);
  a.st = (float2*)(w + L.st);
  a.dsum = (float*)(w + L.dsum);
  a.part = (float*)(w + L.part);
  a.order = (int*)(w + L.order);
  a.nch = L.nch;
  a.scale = 1.0f / sqrtf((float)s.hd);
  return a;
}

static void transpose_kv(hipStream_t st, const uint16_t* src, int nrows, int cols, int ld, uint16_t* dst) {
  hipLaunchKernelGGL(k_tr_kv_t, dim3((ld + 31) / 32, (cols + 31) / 32), dim3(256), 0, st, src, nrows, cols, ld, dst);
}

template <typename F>
static void by_hd(int hd, F&& f) {
  if (hd == 64) f(std::integral_constant<int, 64>{});
  else f(std::integral_constant<int, 128>{});
}

}  // namespace dflare

using namespace dflare;

extern "C" {

size_t dflare_anchor_attention_workspace(int32_t n_blocks, int32_t B, int32_t T, int32_t n_q, int32_t n_kv,
                                         int32_t hd) {
  if (att_check(n_blocks, B, T, n_q, n_kv, hd) != DFLARE_OK) return 0;
  return ws_layout(att_shape(n_blocks, B, T, n_q, n_kv, hd)).total;
}

int dflare_anchor_attention_fwd(const void* q, const void* k_ctx, const void* v_ctx, const void* k_blk,
                                const void* v_blk, const int32_t* anchors, int32_t n_blocks, int32_t B, int32_t T,
                                int32_t n_q, int32_t n_kv, int32_t hd, float* out, float* lse, void* workspace,
                                size_t workspace_bytes, void* stream) {
  const int rc = att_check(n_blocks, B, T, n_q, n_kv, hd);
  if (rc != DFLARE_OK) return rc;
  if (!q || !k_blk || !v_blk || !anchors || !out || !lse || !workspace || (T > 0 && (!k_ctx || !v_ctx)))
    return DFLARE_ERR_INVALID_ARG;
  const AttnShapeT s = att_shape(n_blocks, B, T, n_q, n_kv, hd);
  if (workspace_bytes < ws_layout(s).total) return DFLARE_ERR_INVALID_ARG;
  hipStream_t st = (hipStream_t)stream;
  AttnT a = att_args(s, q, k_ctx, v_ctx, k_blk, v_blk, anchors, workspace);
  a.out = out;
  a.lse = lse;
  const int cols = n_kv * hd;
  const uint16_t* zero_src = a.kb;  // with T = 0 the context copies are all zeros
  transpose_kv(st, T > 0 ? a.vc : zero_src, T, cols, s.Tp, a.vct);
  hipLaunchKernelGGL(k_tr_blk_t, dim3(n_blocks, (cols + 255) / 256), dim3(256), 0, st, a.vb, n_blocks, B, cols, a.vbt);
  hipLaunchKernelGGL(k_anchor_order, dim3((n_blocks + 63) / 64), dim3(256), 0, st, anchors, n_blocks, T, a.order);
  const bool two = (s.R + 15) / 16 > 4;
  by_hd(hd, [&](auto h) {
    constexpr int HD = decltype(h)::value;
    if (two) hipLaunchKernelGGL((k_aatt_rows<HD, false, 2>), dim3(n_blocks, n_kv), dim3(kTrT), 0, st, a);
    else hipLaunchKernelGGL((k_aatt_rows<HD, false, 1>), dim3(n_blocks, n_kv), dim3(kTrT), 0, st, a);
  });
  return hipGetLastError() == hipSuccess ? DFLARE_OK : DFLARE_ERR_HIP;
}

int dflare_anchor_attention_bwd(const void* q, const void* k_ctx, const void* v_ctx, const void* k_blk,
                                const void* v_blk, const int32_t* anchors, int32_t n_blocks, int32_t B, int32_t T,
                                int32_t n_q, int32_t n_kv, int32_t hd, const float* out, const float* lse,
                                const float* dout, float* dq, float* dk_ctx, float* dv_ctx, float* dk_blk,
                                float* dv_blk, void* workspace, size_t workspace_bytes, void* stream) {
  const int rc = att_check(n_blocks, B, T, n_q, n_kv, hd);
  if (rc != DFLARE_OK) return rc;
  if (!q || !k_blk || !v_blk || !anchors || !out || !lse || !dout || !dq || !dk_blk || !dv_blk || !workspace ||
      (T > 0 && (!k_ctx || !v_ctx || !dk_ctx || !dv_ctx)))
    return DFLARE_ERR_INVALID_ARG;
  const AttnShapeT s = att_shape(n_blocks, B, T, n_q, n_kv, hd);
  if (workspace_bytes < ws_layout(s).total) return DFLARE_ERR_INVALID_ARG;
  hipStream_t st = (hipStream_t)stream;
  AttnT a = att_args(s, q, k_ctx, v_ctx, k_blk, v_blk, anchors, workspace);
  a.out = nullptr;
  a.lse = const_cast<float*>(lse);
  a.dout = dout;
  a.dq = dq;
  a.dkc = dk_ctx;
  a.dvc = dv_ctx;
  a.dkb = dk_blk;
  a.dvb = dv_blk;
  const int cols = n_kv * hd;
  const uint16_t* zero_src = a.kb;
  transpose_kv(st, T > 0 ? a.kc : zero_src, T, cols, s.Tp, a.kct);
  hipLaunchKernelGGL(k_tr_blk_t, dim3(n_blocks, (cols + 255) / 256), dim3(256), 0, st, a.kb, n_blocks, B, cols, a.kbt);
  hipLaunchKernelGGL(k_anchor_order, dim3((n_blocks + 63) / 64), dim3(256), 0, st, anchors, n_blocks, T, a.order);
  by_hd(hd, [&](auto h) {
    constexpr int HD = decltype(h)::value;
    hipLaunchKernelGGL((k_bwd_prep<HD>), dim3(n_blocks, n_kv), dim3(256), (size_t)4 * HD * s.Rp, st, a.q, dout, out,
                       (const float*)a.lse, s, a.dob, a.dsum, a.qr, a.dor, a.st, a.qt, a.dot);
    if ((s.R + 15) / 16 > 4) hipLaunchKernelGGL((k_aatt_rows<HD, true, 2>), dim3(n_blocks, n_kv), dim3(kTrT), 0, st, a);
    else hipLaunchKernelGGL((k_aatt_rows<HD, true, 1>), dim3(n_blocks, n_kv), dim3(kTrT), 0, st, a);
    hipLaunchKernelGGL((k_aatt_kvb<HD>), dim3(n_blocks, n_kv, 1), dim3(kTrT), 0, st, a);
    if (T > 0) hipLaunchKernelGGL((k_aatt_kvc<HD>), dim3((T + 63) / 64, n_kv, a.nch), dim3(kTrT), 0, st, a);
  });
  if (T > 0) {
    const long n = (long)T * n_kv * hd;
    hipLaunchKernelGGL(k_aatt_sum, dim3((int)std::min<long>((n + 255) / 256, 4096)), dim3(256), 0, st, a.part, a.nch,
                       n, dk_ctx, dv_ctx);
  }
  return hipGetLastError() == hipSuccess ? DFLARE_OK : DFLARE_ERR_HIP;
}

size_t dflare_weighted_ce_workspace(int32_t rows) { return ((size_t)3 * rows + 64) * 4; }

}  // extern "C"

namespace {

// The four launches of the weighted CE; w holds at least rows + 1 floats (the row weights,
// then 1 / sum w), every one written by the first launch before any other reads it.
void launch_weighted_ce(hipStream_t st, const float* logits, const int32_t* labels, int32_t rows, int32_t V,
                        int32_t B, float gamma, float* loss, float* row_ce, float* dlogits, float* w) {
  float* inv = w + rows;
  hipLaunchKernelGGL(k_wce_weights, dim3(1), dim3(256), 0, st, labels, rows, V, B, gamma, w, inv);
  if (V % 4 == 0 && (long)V >= kCeOMin && (long)V <= kCeOCap)
    hipLaunchKernelGGL(k_wce_chip, dim3(std::min(rows, kCeRows)), dim3(kCeOT), 0, st, logits, labels, rows, V, B,
                       (const float*)w, (const float*)inv, row_ce, dlogits);
  else
    hipLaunchKernelGGL(k_wce_fused, dim3(std::min(rows, kCeRows)), dim3(kCeT), 0, st, logits, labels, rows, V, B,
                       (const float*)w, (const float*)inv, row_ce, dlogits);
  hipLaunchKernelGGL(k_wce_loss, dim3(1), dim3(256), 0, st, w, row_ce, rows, loss);
}

bool ce_args_ok(const float* logits, const int32_t* labels, int32_t rows, int32_t V, int32_t B, float gamma,
                const float* loss, const float* row_ce, const float* dlogits) {
  return logits && labels && loss && row_ce && dlogits && rows >= 1 && V >= 1 && B >= 1 && rows % B == 0 &&
         gamma > 0.f && isfinite(gamma);
}

// Scratch of the allocation-free weighted CE: the row weights and 1 / sum w of one call.
// Each GPU the library runs on holds its own copy until the process ends.  In host code the
// array's name is not a device address: kernels get the address hipGetSymbolAddress returns
// for the current device, looked up once per device.
constexpr int kCeNoAllocMaxRows = DFLARE_WEIGHTED_CE_NOALLOC_MAX_ROWS;
__device__ __align__(256) float scratch[kCeNoAllocMaxRows + 64];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch[kMaxDevices];

// address of this device's scratch array (the device of `st`, which must be current)
int scratch_address(hipStream_t st, float** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return DFLARE_ERR_HIP;
  if (st) {
    int sdev = -1;
    if (hipStreamGetDevice(st, &sdev) != hipSuccess) return DFLARE_ERR_HIP;
    if (sdev != dev) return DFLARE_ERR_INVALID_ARG;
  }
  if (dev < 0 || dev >= kMaxDevices) return DFLARE_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return DFLARE_ERR_HIP;
    g_scratch[dev] = static_cast<float*>(p);
  }
  *out = g_scratch[dev];
  return DFLARE_OK;
}

}  // namespace

extern "C" {

int dflare_weighted_ce(const float* logits, const int32_t* labels, int32_t rows, int32_t V, int32_t B, float gamma,
                       float* loss, float* row_ce, float* dlogits, void* workspace, size_t workspace_bytes,
                       void* stream) {
  if (!ce_args_ok(logits, labels, rows, V, B, gamma, loss, row_ce, dlogits) || !workspace)
    return DFLARE_ERR_INVALID_ARG;
  if (workspace_bytes < dflare_weighted_ce_workspace(rows)) return DFLARE_ERR_INVALID_ARG;
  launch_weighted_ce((hipStream_t)stream, logits, labels, rows, V, B, gamma, loss, row_ce, dlogits,
                     static_cast<float*>(workspace));
  return hipGetLastError() == hipSuccess ? DFLARE_OK : DFLARE_ERR_HIP;
}

int dflare_weighted_ce_noalloc(const float* logits, const int32_t* labels, int32_t rows, int32_t V, int32_t B,
                               float gamma, float* loss, float* row_ce, float* dlogits, void* stream) {
  if (!ce_args_ok(logits, labels, rows, V, B, gamma, loss, row_ce, dlogits)) return DFLARE_ERR_INVALID_ARG;
  if (rows > kCeNoAllocMaxRows) return DFLARE_ERR_INVALID_ARG;
  hipStream_t st = (hipStream_t)stream;
  float* w = nullptr;
  const int rc = scratch_address(st, &w);
  if (rc != DFLARE_OK) return rc;
  launch_weighted_ce(st, logits, labels, rows, V, B, gamma, loss, row_ce, dlogits, w);
  return hipGetLastError() == hipSuccess ? DFLARE_OK : DFLARE_ERR_HIP;
}

}  // extern "C"
