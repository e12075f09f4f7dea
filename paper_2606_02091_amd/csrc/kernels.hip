// HIP kernels of the DFlare draft step for gfx950 (CDNA4, wave64, MFMA).
//
// Data types: weights, embeddings and the KV cache are bf16; activations, the
// residual stream and every accumulation are fp32.  Activations enter the bf16
// matrix cores as an exact-sum pair hi + lo of bf16 values (hi = bf16(x),
// lo = bf16(x - hi)), so each product carries about 16 mantissa bits of the
// activation against the exact bf16 weight; the doubled MFMA work is free
// because every GEMM here streams its weights from HBM (batch-1, 16 rows).
#include "dflare_impl.h"

#include <math.h>

namespace dflare {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf2f(uint32_t b) { return __uint_as_float(b << 16); }

// float -> bf16 bits, round to nearest even (inputs are finite).
__device__ __forceinline__ uint32_t f2bf(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ void split_pack8(const float* v, u32x4& hi, u32x4& lo) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    uint32_t h0 = f2bf(v[2 * e]), h1 = f2bf(v[2 * e + 1]);
    uint32_t l0 = f2bf(v[2 * e] - bf2f(h0)), l1 = f2bf(v[2 * e + 1] - bf2f(h1));
    hi[e] = h0 | (h1 << 16);
    lo[e] = l0 | (l1 << 16);
  }
}

// Activations handed from one kernel to the next are stored directly in the A-operand
// layout of v_mfma_f32_16x16x32_bf16, as two bf16 planes hi and lo (x ~= hi + lo):
//   element (row, k) of a [rows, K] matrix sits in 16-row tile row/16, k-tile k/32,
//   lane (row % 16) + 16 * ((k % 32) / 8), slot k % 8; a (row-tile, k-tile) is 1 KiB.
__device__ __forceinline__ long frag_off(int row, int k, int Kt) {
  return ((((long)(row >> 4) * Kt + (k >> 5)) * 64 + (row & 15) + ((k & 31) >> 3) * 16) << 3) + (k & 7);
}

// store the hi/lo planes of two consecutive elements (k even) as one 32-bit word each
__device__ __forceinline__ void store_frag_pair(uint32_t* hi, uint32_t* lo, int row, int k, int Kt, float v0,
                                                float v1) {
  const uint32_t h0 = f2bf(v0), h1 = f2bf(v1);
  const uint32_t l0 = f2bf(v0 - bf2f(h0)), l1 = f2bf(v1 - bf2f(h1));
  const long o = frag_off(row, k, Kt) >> 1;
  hi[o] = h0 | (h1 << 16);
  lo[o] = l0 | (l1 << 16);
}

__device__ __forceinline__ f32x4 mfma(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// ------------------------------------------------------------------------------------------
// init-time helpers
// ------------------------------------------------------------------------------------------

// Pack rows of W[n_src_rows, K] (bf16, row-major) into MFMA B-operand tiles.
__global__ void k_pack(u32x4* dst, const uint16_t* __restrict__ src0, const uint16_t* __restrict__ src1,
                       int n_src_rows, int K, int nt_begin, int nt_count, int Kt_total, int mode, int hd) {
  const int Kt = K / 32;
  const long total = (long)nt_count * Kt * 64;
  for (long idx = blockIdx.x * (long)blockDim.x + threadIdx.x; idx < total;
       idx += (long)gridDim.x * blockDim.x) {
    const int lane = (int)(idx & 63);
    const long tile = idx >> 6;
    const int kt = (int)(tile % Kt);
    const int nt = (int)(tile / Kt);
    const int p = nt * 16 + (lane & 15);  // packed output column inside this region
    const int c = lane & 15;
    const uint16_t* src = src0;
    int row = p;
    if (mode == PACK_ROPE) {
      const int tph = hd / 16, head = nt / tph, j = nt % tph;
      const int dim = (c < 8) ? (8 * j + c) : (hd / 2 + 8 * j + (c - 8));
      row = head * hd + dim;
    } else if (mode == PACK_SWIGLU) {
      row = 8 * nt + (c & 7);
      src = (c < 8) ? src0 : src1;
    }
    u32x4 v = {0u, 0u, 0u, 0u};
    if (row < n_src_rows) {
      const uint16_t* s = src + (long)row * K + kt * 32 + (lane >> 4) * 8;
      v = *reinterpret_cast<const u32x4*>(s);
    }
    dst[((long)(nt_begin + nt) * Kt_total + kt) * 64 + lane] = v;
  }
}

__global__ void k_bf16_to_f32(float* dst, const uint16_t* src, long n) {
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x)
    dst[i] = src ? bf2f(src[i]) : 1.0f;
}

// ------------------------------------------------------------------------------------------
// per-call prologue: step parameters and a private copy of the block ids
// ------------------------------------------------------------------------------------------
__global__ void k_prologue(StepParams* p, StepParams host, const int* ids_src, int* ids_dst, int B) {
  const int t = threadIdx.x;
  if (t == 0) {
    p->L = host.L;
    p->n_new = host.n_new;
  }
  if (t < 16) p->pos[t] = host.pos[t];
  if (ids_src && t < B) ids_dst[t] = ids_src[t];
}

// ------------------------------------------------------------------------------------------
// embedding gather: X[b, :] = E[id_b, :] (fp32), per-16-column sums of squares, and the
// A fragments of X * g (g = gain of the first pre-attention RMSNorm)
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_embed(const uint16_t* __restrict__ E, const int* __restrict__ ids,
                                               int vocab, int H, float* X, float* stats,
                                               const float* __restrict__ gain, u32x4* a_hi, u32x4* a_lo) {
  const int b = blockIdx.x;
  int id = ids[b];
  id = id < 0 ? 0 : (id >= vocab ? vocab - 1 : id);
  const uint16_t* row = E + (long)id * H;
  const int Kt = H / 32;
  for (int k0 = threadIdx.x * 8; k0 < H; k0 += blockDim.x * 8) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(row + k0);
    float f[8], y[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[2 * e] = bf2f(v[e] & 0xFFFFu);
      f[2 * e + 1] = bf2f(v[e] >> 16);
    }
    float sq = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      sq += f[e] * f[e];
      y[e] = f[e] * gain[k0 + e];
    }
    float* xo = X + (long)b * H + k0;
    *reinterpret_cast<float4*>(xo) = make_float4(f[0], f[1], f[2], f[3]);
    *reinterpret_cast<float4*>(xo + 4) = make_float4(f[4], f[5], f[6], f[7]);
    u32x4 hi, lo;
    split_pack8(y, hi, lo);
    const long fo = frag_off(b, k0, Kt) >> 3;
    a_hi[fo] = hi;
    a_lo[fo] = lo;
    sq += __shfl_xor(sq, 1);
    if ((threadIdx.x & 1) == 0) stats[(long)b * (H / 16) + k0 / 16] = sq;
  }
}

// ------------------------------------------------------------------------------------------
// layer fusion (Eq. 3): u^(i)[r, k] = sum_j alpha[i, j] h^(j)[r, k], accumulated in j order.
// Block (512 columns, row r, draft layer i); a lane owns 8 columns and keeps twelve 16-byte
// loads in flight.  Writes the A fragments of u^(i) * g_fuse^(i) and per-16-column sums of
// squares of u^(i); the 1/rms of Eq. 3 is applied in the K/V projection.  The S target rows
// are read from HBM once; the blocks of the other draft layers find them in L2.
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(64) void k_fuse(const uint16_t* __restrict__ hidden, int n, int S, int H,
                                             const float* __restrict__ alpha, const float* __restrict__ gain,
                                             float* ustats, u32x4* ua_hi, u32x4* ua_lo, int n_max, int mt_max,
                                             StepParams* params, int L) {
  const int lane = threadIdx.x;
  const int r = blockIdx.y, i = blockIdx.z;
  if (blockIdx.x == 0 && r == 0 && i == 0 && lane == 0) {  // step parameters for the K/V projection
    params->L = L;
    params->n_new = n;
  }
  const int k0 = blockIdx.x * 512 + lane * 8;
  const bool ok = k0 < H;
  const int Kt = H / 32;
  float u[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int j0 = 0; j0 < S; j0 += 12) {
    u32x4 v[12];
#pragma unroll
    for (int qq = 0; qq < 12; ++qq) {
      v[qq] = u32x4{0u, 0u, 0u, 0u};
      if (ok && j0 + qq < S) v[qq] = *reinterpret_cast<const u32x4*>(hidden + ((long)(j0 + qq) * n + r) * H + k0);
    }
#pragma unroll
    for (int qq = 0; qq < 12; ++qq) {
      if (j0 + qq < S) {
        const float a = alpha[i * S + j0 + qq];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          u[2 * e] = fmaf(a, bf2f(v[qq][e] & 0xFFFFu), u[2 * e]);
          u[2 * e + 1] = fmaf(a, bf2f(v[qq][e] >> 16), u[2 * e + 1]);
        }
      }
    }
  }
  float sq = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) sq += u[e] * u[e];
  sq += __shfl_xor(sq, 1);
  if (ok) {
    float y[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) y[e] = u[e] * gain[(long)i * H + k0 + e];
    u32x4 hi, lo;
    split_pack8(y, hi, lo);
    const long fo = ((long)i * mt_max * Kt * 64 * 8 + frag_off(r, k0, Kt)) >> 3;
    ua_hi[fo] = hi;
    ua_lo[fo] = lo;
    if ((lane & 1) == 0) ustats[((long)i * n_max + r) * (H / 16) + k0 / 16] = sq;
  }
}

// debug: materialise f^(i) = (hi + lo) * rstd, [D, n, H] fp32 (the gain is already applied)
__global__ void k_fused_rows(const u32x4* ua_hi, const u32x4* ua_lo, const float* ustats, int n, int H, int D,
                             int n_max, int mt_max, float eps, float* out) {
  const int r = blockIdx.x, i = blockIdx.y;
  const int Kt = H / 32;
  __shared__ float s_r;
  if (threadIdx.x == 0) {
    float s = 0.f;
    for (int t = 0; t < H / 16; ++t) s += ustats[((long)i * n_max + r) * (H / 16) + t];
    s_r = rsqrtf(s / H + eps);
  }
  __syncthreads();
  const uint16_t* hi = reinterpret_cast<const uint16_t*>(ua_hi);
  const uint16_t* lo = reinterpret_cast<const uint16_t*>(ua_lo);
  for (int k = threadIdx.x; k < H; k += blockDim.x) {
    const long o = (long)i * mt_max * Kt * 64 * 8 + frag_off(r, k, Kt);
    out[((long)i * n + r) * H + k] = (bf2f(hi[o]) + bf2f(lo[o])) * s_r;
  }
}

// ------------------------------------------------------------------------------------------
// weight-streaming GEMM, y[M<=16 per m-tile, N] = x[M, K] W^T.
// Block `group` owns output tiles [group*NT, +NT) over the whole K; its WAVES waves split the
// k range, each streaming its NT weight tiles per k-tile from HBM together with the A
// fragments of the same k-tile (hi and lo planes, from L2: they are shared by every block).
// Two register sets alternate so that one batch of loads is always in flight while the
// previous batch goes through the matrix cores.  The waves' partial sums are added in LDS in
// wave order (fixed, so results do not depend on timing), and wave w < NT then holds output
// tile group*NT + w for the epilogue.  No block ever waits on another: there is no split-K
// across blocks, because making partial sums of one XCD visible to another takes agent-scope
// fences that write back and invalidate the L2 -- far costlier than these kernels.
// ------------------------------------------------------------------------------------------
template <int NT, int WAVES, int EPI>
__global__ __launch_bounds__(64 * WAVES) void k_gemm(GemmArgs a) {
  constexpr int U = 2;  // k-tiles per batch
  __shared__ f32x4 red[WAVES][NT][64];
  __shared__ float s_rstd[16];
  __shared__ float s_bv[NT][16];
  __shared__ int s_bi[NT][16];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int quad = lane >> 4, col = lane & 15;
  const int groups = gridDim.x;
  const int group = blockIdx.x;
  const int layer = blockIdx.y, mt = blockIdx.z;
  const int M = (EPI == EPI_KVT) ? a.e.params->n_new : a.M;
  if (mt * 16 >= M) return;  // whole m-tile idle: every block of it leaves together

  const int kw0 = (a.Kt * wave) / WAVES;
  const int nk = (a.Kt * (wave + 1)) / WAVES - kw0;
  const int nb = (nk + U - 1) / U;
  const int nb2 = (nb + 1) & ~1;
  const int nt0 = group * NT;

  // Tile addresses; a tile past the wave's range or a padding output tile reads the zero
  // tile instead, so the streaming loop has no branches.
  const u32x4* zt = a.zero + lane;
  const u32x4* Wl = a.W + layer * a.w_layer_stride;
  const u32x4* wrow[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) wrow[j] = Wl + ((long)(nt0 + j) * a.Kt + kw0) * 64 + lane;
  const long abase = layer * a.a_layer_stride + ((long)mt * a.Kt + kw0) * 64 + lane;
  const u32x4* ah_row = a.Ahi + abase;
  const u32x4* al_row = a.Alo + abase;
  auto wptr = [&](int j, int t) -> const u32x4* {
    return (t < nk && nt0 + j < a.Nt) ? wrow[j] + (long)t * 64 : zt;
  };
  auto ahp = [&](int t) -> const u32x4* { return (t < nk) ? ah_row + (long)t * 64 : zt; };
  auto alp = [&](int t) -> const u32x4* { return (t < nk) ? al_row + (long)t * 64 : zt; };

  u32x4 wA[U][NT], hA[U], lA[U], wB[U][NT], hB[U], lB[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
#pragma unroll
    for (int j = 0; j < NT; ++j) wA[u][j] = __builtin_nontemporal_load(wptr(j, u));
    hA[u] = *ahp(u);
    lA[u] = *alp(u);
  }
#pragma unroll
  for (int u = 0; u < U; ++u) {
#pragma unroll
    for (int j = 0; j < NT; ++j) wB[u][j] = __builtin_nontemporal_load(wptr(j, U + u));
    hB[u] = *ahp(U + u);
    lB[u] = *alp(U + u);
  }
  f32x4 acc_h[NT], acc_l[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    acc_h[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    acc_l[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  for (int b = 0; b < nb2; b += 2) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        acc_h[j] = mfma(hA[u], wA[u][j], acc_h[j]);
        acc_l[j] = mfma(lA[u], wA[u][j], acc_l[j]);
      }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = (b + 2) * U + u;
#pragma unroll
      for (int j = 0; j < NT; ++j) wA[u][j] = __builtin_nontemporal_load(wptr(j, t));
      hA[u] = *ahp(t);
      lA[u] = *alp(t);
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        acc_h[j] = mfma(hB[u], wB[u][j], acc_h[j]);
        acc_l[j] = mfma(lB[u], wB[u][j], acc_l[j]);
      }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = (b + 3) * U + u;
#pragma unroll
      for (int j = 0; j < NT; ++j) wB[u][j] = __builtin_nontemporal_load(wptr(j, t));
      hB[u] = *ahp(t);
      lB[u] = *alp(t);
    }
  }

  // waves -> tiles: wave w < NT receives tile w summed over the waves in wave order
#pragma unroll
  for (int j = 0; j < NT; ++j) red[wave][j][lane] = acc_h[j] + acc_l[j];
  __syncthreads();
  const bool owner = wave < NT;
  const int nt = nt0 + (owner ? wave : 0);
  const bool has_tile = owner && nt < a.Nt;  // wave-uniform
  f32x4 v = {0.f, 0.f, 0.f, 0.f};
  if (owner) {
    v = red[0][wave][lane];
#pragma unroll
    for (int w = 1; w < WAVES; ++w) v += red[w][wave][lane];
  }

  // 1/rms of the rows (RMSNorm consumers): (x*g/rms) W^T = (1/rms) (x*g) W^T
  if (a.stats) {
    if (tid < 256) {
      const int row = tid >> 4, part = tid & 15;
      float s = 0.f;
      if (mt * 16 + row < M) {
        const float* st = a.stats + layer * a.stats_layer_stride + (long)(mt * 16 + row) * a.n_stat;
#pragma unroll
        for (int q = 0; q < 32; ++q) {
          const int t = part + 16 * q;
          if (t < a.n_stat) s += st[t];
        }
      }
      s += __shfl_xor(s, 8);
      s += __shfl_xor(s, 4);
      s += __shfl_xor(s, 2);
      s += __shfl_xor(s, 1);
      if (part == 0) s_rstd[row] = rsqrtf(s * a.inv_dim + a.eps);
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] *= s_rstd[quad * 4 + i];
  }

  // epilogues.  The owner lane holds rows mt*16 + 4*quad + i (i < 4) of output column nt*16 + col.
  const EpiArgs& e = a.e;
  if constexpr (EPI == EPI_RESID) {
    if (has_tile) {
      const int k = nt * 16 + col;
      const float gn = e.next_gain[k];
      float sq[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = mt * 16 + quad * 4 + i;
        float x = 0.f;
        if (row < M) {
          float* p = e.out + (long)row * e.ldo + k;
          x = *p + v[i];
          *p = x;
        }
        sq[i] = x * x;
        const float y = x * gn;
        const float y1 = __shfl_xor(y, 1);
        if ((col & 1) == 0 && row < M) store_frag_pair(e.na_hi, e.na_lo, row, k, e.na_Kt, y, y1);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        sq[i] += __shfl_xor(sq[i], 1);
        sq[i] += __shfl_xor(sq[i], 2);
        sq[i] += __shfl_xor(sq[i], 4);
        sq[i] += __shfl_xor(sq[i], 8);
      }
      if (col == 0)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = mt * 16 + quad * 4 + i;
          if (row < M) e.stats_out[(long)row * e.n_stat_out + nt] = sq[i];
        }
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    if (has_tile) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float g = v[i];
        const float up = __shfl_xor(g, 8);
        const float hv = (col < 8) ? g / (1.0f + expf(-g)) * up : 0.f;
        const float h1 = __shfl_xor(hv, 1);
        const int row = mt * 16 + quad * 4 + i;
        if (col < 8 && (col & 1) == 0 && row < M) store_frag_pair(e.na_hi, e.na_lo, row, nt * 8 + col, e.na_Kt, hv, h1);
      }
    }
  } else if constexpr (EPI == EPI_QKV || EPI == EPI_KVT) {
    if (has_tile) {
      const int L = e.params->L;
      const int tph = e.hd / 16, half = e.hd / 2;
      uint16_t* kc = e.kc + (EPI == EPI_KVT ? layer * e.cache_layer_stride : 0);
      uint16_t* vt = e.vt + (EPI == EPI_KVT ? layer * e.cache_layer_stride : 0);
      int region, t;  // 0 = Q, 1 = K, 2 = V
      if (nt < e.q_tiles) { region = 0; t = nt; }
      else if (nt < e.q_tiles + e.kv_tiles) { region = 1; t = nt - e.q_tiles; }
      else { region = 2; t = nt - e.q_tiles - e.kv_tiles; }
      const int head = t / tph, jj = t % tph;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = mt * 16 + quad * 4 + i;
        const bool valid = (EPI == EPI_QKV) ? (row < e.B) : (row < M);
        const int pos = valid ? ((EPI == EPI_QKV) ? e.params->pos[row] : L + row) : 0;
        const int slot = L + row;
        const float x = v[i];
        const float partner = __shfl_xor(x, 8);
        if (region < 2) {
          const int m = 8 * jj + (col & 7);
          const int dim = (col < 8) ? m : half + m;
          const float2 cs = e.rope[(long)pos * half + m];
          const float y = (col < 8) ? (x * cs.x - partner * cs.y) : (x * cs.x + partner * cs.y);
          if (valid) {
            if (region == 0) {
              e.out[(long)row * e.ldo + head * e.hd + dim] = y;
            } else {  // the cache keeps y as two bf16 planes, y ~= hi + lo
              const long ix = ((long)head * e.Lcap + slot) * e.hd + dim;
              const uint32_t hb = f2bf(y);
              kc[ix] = (uint16_t)hb;
              kc[ix + e.plane] = (uint16_t)f2bf(y - bf2f(hb));
            }
          }
        } else if (valid) {
          const int dim = jj * 16 + col;
          const long ix = ((long)head * e.hd + dim) * e.Lcap + slot;
          const uint32_t hb = f2bf(x);
          vt[ix] = (uint16_t)hb;
          vt[ix + e.plane] = (uint16_t)f2bf(x - bf2f(hb));
        }
      }
    }
  } else if constexpr (EPI == EPI_ARGMAX) {
    if (owner) {
      const int c = nt * 16 + col;
      const bool ok = has_tile && c < e.vocab;
      float bv[4];
      int bi[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = quad * 4 + i;
        if (ok && e.logits && row < e.B) e.logits[(long)row * e.vocab + c] = v[i];
        bv[i] = ok ? v[i] : -INFINITY;
        bi[i] = ok ? c : 0x7FFFFFFF;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) {
          const float ov = __shfl_xor(bv[i], off);
          const int oi = __shfl_xor(bi[i], off);
          if (ov > bv[i] || (ov == bv[i] && oi < bi[i])) { bv[i] = ov; bi[i] = oi; }
        }
      if (col == 0)
#pragma unroll
        for (int i = 0; i < 4; ++i) { s_bv[wave][quad * 4 + i] = bv[i]; s_bi[wave][quad * 4 + i] = bi[i]; }
    }
    __syncthreads();
    if (tid < 16) {  // this block's best per row; the combine kernel picks across blocks
      float bvv = s_bv[0][tid];
      int ix = s_bi[0][tid];
      for (int w = 1; w < NT; ++w) {
        const float ov = s_bv[w][tid];
        const int oi = s_bi[w][tid];
        if (ov > bvv || (ov == bvv && oi < ix)) { bvv = ov; ix = oi; }
      }
      e.pmax[(long)tid * groups + group] = bvv;
      e.pidx[(long)tid * groups + group] = ix;
    }
  }
}

// per-row argmax over the blocks' partial results (ties: lowest token id)
__global__ __launch_bounds__(256) void k_argmax_combine(const float* pmax, const int* pidx, int groups,
                                                        int* tokens) {
  __shared__ float s_v[4];
  __shared__ int s_i[4];
  const int row = blockIdx.x, tid = threadIdx.x;
  float v = -INFINITY;
  int ix = 0x7FFFFFFF;
  for (int g = tid; g < groups; g += 256) {
    const float ov = pmax[(long)row * groups + g];
    const int oi = pidx[(long)row * groups + g];
    if (ov > v || (ov == v && oi < ix)) { v = ov; ix = oi; }
  }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const float ov = __shfl_xor(v, off);
    const int oi = __shfl_xor(ix, off);
    if (ov > v || (ov == v && oi < ix)) { v = ov; ix = oi; }
  }
  if ((tid & 63) == 0) {
    s_v[tid >> 6] = v;
    s_i[tid >> 6] = ix;
  }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < 4; ++w)
      if (s_v[w] > v || (s_v[w] == v && s_i[w] < ix)) { v = s_v[w]; ix = s_i[w]; }
    tokens[row] = (ix == 0x7FFFFFFF) ? 0 : ix;
  }
}

// ------------------------------------------------------------------------------------------
// block attention, split over the key axis (Sec. 3.2: no mask, every block row sees the
// whole context and the whole block).  Block (chunk c, KV head g) of 8 waves: chunk c holds
// keys [c*CK, (c+1)*CK) of the context, the last chunk also the B block keys (cache slots
// L..L+B-1).  K rows and V^T rows of the chunk, both bf16 planes (hi, lo), are copied to LDS
// with every load in flight at once (16-byte pieces, XOR-swizzled columns so that the
// fragment reads of 16 different rows hit different banks).  Wave w then takes query tile w:
// rows r = w*16 + lane%16 of the G*B rows that share head g (r -> query head g*G + r/B, block
// position r%B).  Scores are formed transposed, S^T = K Q^T, so that the probabilities land in
// exactly the B-operand layout of the P V product and never leave registers.  Products of
// two hi/lo pairs keep the three terms above 2^-16 relative: hi*hi + hi*lo + lo*hi.
// ------------------------------------------------------------------------------------------
template <int HD, int CK>
__global__ __launch_bounds__(512) void k_attn(AttnArgs a) {
  constexpr int CKM = CK + 32;   // keys held by a block (room for the B <= 16 block keys)
  constexpr int KC = HD / 8;     // 16-byte columns of a K row
  constexpr int VC = CKM / 8;    // 16-byte columns of a V^T row (a multiple of 4)
  constexpr int KPC = 2 * CKM * KC, VPC = 2 * HD * VC;  // pieces of both planes
  constexpr int PER = (KPC + VPC) / 512;                 // pieces per thread
  static_assert(KPC % 512 == 0 && VPC % 512 == 0, "piece counts must split evenly over the block");
  __shared__ u32x4 sK[2][CKM * KC];  // (row r, column c) at r*KC + (c ^ (r & 7))
  __shared__ u32x4 sV[2][HD * VC];   // (row d, column c) at d*VC + (c ^ (d & 3))
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int quad = lane >> 4, q = lane & 15;
  const int g = blockIdx.y, c = blockIdx.x;
  const int L = a.params->L;
  const int nch = max(1, (L + CK - 1) / CK);
  if (c >= nch) return;
  const int kbeg = c * CK;
  const int kend = (c == nch - 1) ? L + a.B : kbeg + CK;
  const int nkeys = kend - kbeg;  // <= CK + B
  const int G = a.n_q / a.n_kv;
  const int R = G * a.B;

  // 1. issue every piece of the chunk and this wave's query row
  u32x4 pc[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int p = i * 512 + tid;
    pc[i] = u32x4{0u, 0u, 0u, 0u};
    if (p < KPC) {  // uniform for a given i
      const int pl = p / (CKM * KC), rem = p % (CKM * KC);
      const int r = rem / KC, col = rem % KC;
      if (r < nkeys)
        pc[i] = *reinterpret_cast<const u32x4*>(a.kc + pl * a.plane + ((long)g * a.Lcap + kbeg + r) * HD + col * 8);
    } else {
      const int pv = p - KPC;
      const int pl = pv / (HD * VC), rem = pv % (HD * VC);
      const int d = rem / VC, col = rem % VC;
      if (col * 8 < nkeys)
        pc[i] = *reinterpret_cast<const u32x4*>(a.vt + pl * a.plane + ((long)g * HD + d) * a.Lcap + kbeg + col * 8);
    }
  }
  const int r = w * 16 + q;
  const bool active = w * 16 < R;  // wave-uniform
  const bool rv = r < R;
  float4 qx[HD / 16];
  {
    const int b = rv ? r % a.B : 0;
    const int h = g * G + (rv ? r / a.B : 0);
#pragma unroll
    for (int ks = 0; ks < HD / 32; ++ks) {
      const float* src = a.Q + (long)b * a.q_dim + h * HD + ks * 32 + quad * 8;
      qx[2 * ks] = (active && rv) ? *reinterpret_cast<const float4*>(src) : make_float4(0.f, 0.f, 0.f, 0.f);
      qx[2 * ks + 1] = (active && rv) ? *reinterpret_cast<const float4*>(src + 4) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
  // 2. pieces to LDS (keys past the end become zeros)
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int p = i * 512 + tid;
    if (p < KPC) {
      const int pl = p / (CKM * KC), rem = p % (CKM * KC);
      const int rr = rem / KC, col = rem % KC;
      sK[pl][rr * KC + (col ^ (rr & 7))] = pc[i];
    } else {
      const int pv = p - KPC;
      const int pl = pv / (HD * VC), rem = pv % (HD * VC);
      const int d = rem / VC, col = rem % VC;
      u32x4 v = pc[i];
      const int nv = nkeys - col * 8;  // valid keys in this piece
      if (nv < 8) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (2 * e >= nv) v[e] = 0u;
          else if (2 * e + 1 >= nv) v[e] &= 0xFFFFu;
        }
      }
      sV[pl][d * VC + (col ^ (d & 3))] = v;
    }
  }
  __syncthreads();
  if (!active) return;

  u32x4 qh[HD / 32], ql[HD / 32];
#pragma unroll
  for (int ks = 0; ks < HD / 32; ++ks) {
    const float4 x0 = qx[2 * ks], x1 = qx[2 * ks + 1];
    float v[8] = {x0.x * a.qscale, x0.y * a.qscale, x0.z * a.qscale, x0.w * a.qscale,
                  x1.x * a.qscale, x1.y * a.qscale, x1.z * a.qscale, x1.w * a.qscale};
    split_pack8(v, qh[ks], ql[ks]);
  }
  f32x4 s[CKM / 16];
#pragma unroll
  for (int kt = 0; kt < CKM / 16; ++kt) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    const int rr = kt * 16 + q;
#pragma unroll
    for (int ks = 0; ks < HD / 32; ++ks) {
      const int slot = rr * KC + ((ks * 4 + quad) ^ (rr & 7));
      const u32x4 kh = sK[0][slot], kl = sK[1][slot];
      acc = mfma(kh, qh[ks], acc);
      acc = mfma(kh, ql[ks], acc);
      acc = mfma(kl, qh[ks], acc);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (kt * 16 + quad * 4 + i >= nkeys) acc[i] = -INFINITY;
    s[kt] = acc;
  }
  // softmax statistics per query row (column q), in the log2 domain
  float m = -INFINITY;
#pragma unroll
  for (int kt = 0; kt < CKM / 16; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i) m = fmaxf(m, s[kt][i]);
  m = fmaxf(m, __shfl_xor(m, 16));
  m = fmaxf(m, __shfl_xor(m, 32));
  float l = 0.f;
#pragma unroll
  for (int kt = 0; kt < CKM / 16; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float p = exp2f(s[kt][i] - m);
      s[kt][i] = p;
      l += p;
    }
  l += __shfl_xor(l, 16);
  l += __shfl_xor(l, 32);
  // O^T = V^T P^T over the chunk
  f32x4 o[HD / 16];
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  const u32x2* v2h = reinterpret_cast<const u32x2*>(sV[0]);
  const u32x2* v2l = reinterpret_cast<const u32x2*>(sV[1]);
#pragma unroll
  for (int kk = 0; kk < CKM / 32; ++kk) {
    float pv[8] = {s[2 * kk][0], s[2 * kk][1], s[2 * kk][2], s[2 * kk][3],
                   s[2 * kk + 1][0], s[2 * kk + 1][1], s[2 * kk + 1][2], s[2 * kk + 1][3]};
    u32x4 ph, pl;
    split_pack8(pv, ph, pl);
    const int c0 = kk * 4 + (quad >> 1), half = quad & 1;  // keys kk*32 + 4*quad + 0..3 (+16)
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) {
      const int d = dt * 16 + q;
      const int i0 = (d * VC + (c0 ^ (d & 3))) * 2 + half;
      const int i1 = (d * VC + ((c0 + 2) ^ (d & 3))) * 2 + half;
      const u32x2 h0 = v2h[i0], h1 = v2h[i1], l0 = v2l[i0], l1 = v2l[i1];
      const u32x4 vh = {h0[0], h0[1], h1[0], h1[1]};
      const u32x4 vl = {l0[0], l0[1], l1[0], l1[1]};
      o[dt] = mfma(vh, ph, o[dt]);
      o[dt] = mfma(vh, pl, o[dt]);
      o[dt] = mfma(vl, ph, o[dt]);
    }
  }
  if (rv) {
    const long base = ((long)c * a.n_kv + g) * a.Rpad + r;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt)
      *reinterpret_cast<f32x4*>(a.opart + base * HD + dt * 16 + quad * 4) = o[dt];
    if (quad == 0) a.ml[base] = make_float2(m, l);
  }
}

// combine the chunk partials of one query row r of KV head g:
// O = sum_c 2^(m_c - M) O_c / sum_c 2^(m_c - M) l_c, written as the A fragments of the output
// projection.  Block (r, g); thread (chunk slot cs, 8 dims d0..d0+7).
template <int HD, int CK>
__global__ __launch_bounds__(256) void k_attn_combine(AttnArgs a) {
  constexpr int DG = HD / 8, CS = 256 / DG;
  __shared__ float s_red[256];
  __shared__ float s_num[CS][HD];
  const int r = blockIdx.x, g = blockIdx.y, tid = threadIdx.x;
  const int G = a.n_q / a.n_kv;
  const int R = G * a.B;
  if (r >= R) return;
  const int nch = max(1, (a.params->L + CK - 1) / CK);  // the last chunk also holds the block keys
  const float2* ml = a.ml + (long)g * a.Rpad + r;  // chunk c at ml[c * n_kv * Rpad]
  const long mstride = (long)a.n_kv * a.Rpad;
  // 1. M = max_c m_c
  float m = -INFINITY;
  for (int c = tid; c < nch; c += 256) m = fmaxf(m, ml[c * mstride].x);
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) m = fmaxf(m, __shfl_xor(m, off));
  if ((tid & 63) == 0) s_red[tid >> 6] = m;
  __syncthreads();
  const float M = fmaxf(fmaxf(s_red[0], s_red[1]), fmaxf(s_red[2], s_red[3]));
  // 2. weighted sums; chunk slots in a fixed order
  const int dg = tid % DG, cs = tid / DG, d0 = dg * 8;
  float num[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float den = 0.f;
#pragma unroll 4
  for (int c = cs; c < nch; c += CS) {
    const float2 mc = ml[c * mstride];
    const float wgt = exp2f(mc.x - M);
    den += wgt * mc.y;
    const float* op = a.opart + (((long)c * a.n_kv + g) * a.Rpad + r) * HD + d0;
    const float4 o0 = *reinterpret_cast<const float4*>(op);
    const float4 o1 = *reinterpret_cast<const float4*>(op + 4);
    num[0] += wgt * o0.x; num[1] += wgt * o0.y; num[2] += wgt * o0.z; num[3] += wgt * o0.w;
    num[4] += wgt * o1.x; num[5] += wgt * o1.y; num[6] += wgt * o1.z; num[7] += wgt * o1.w;
  }
  __syncthreads();
#pragma unroll
  for (int e = 0; e < 8; ++e) s_num[cs][d0 + e] = num[e];
  if (dg == 0) s_red[cs] = den;
  __syncthreads();
  if (tid < DG) {
    float acc[8];
    float dsum = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
    for (int k = 0; k < CS; ++k) {
      dsum += s_red[k];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += s_num[k][tid * 8 + e];
    }
    const float inv = 1.0f / dsum;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] *= inv;
    const int b = r % a.B, h = g * G + r / a.B;
    u32x4 hi, lo;
    split_pack8(acc, hi, lo);
    const long fo = frag_off(b, h * HD + tid * 8, a.oa_Kt) >> 3;
    a.oa_hi[fo] = hi;
    a.oa_lo[fo] = lo;
  }
}

// ------------------------------------------------------------------------------------------
// launchers
// ------------------------------------------------------------------------------------------
void launch_pack(hipStream_t s, u32x4* dst, const uint16_t* src0, const uint16_t* src1, int n_src_rows, int K,
                 int nt_begin, int nt_count, int Kt_total, int mode, int hd) {
  const long total = (long)nt_count * (K / 32) * 64;
  int blocks = (int)((total + 255) / 256);
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_pack, dim3(blocks), dim3(256), 0, s, dst, src0, src1, n_src_rows, K, nt_begin, nt_count,
                     Kt_total, mode, hd);
}

void launch_bf16_to_f32(hipStream_t s, float* dst, const uint16_t* src, long n) {
  int blocks = (int)((n + 255) / 256);
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_bf16_to_f32, dim3(blocks), dim3(256), 0, s, dst, src, n);
}

void launch_prologue(hipStream_t s, StepParams* p, const StepParams& host, const int* ids_src, int* ids_dst,
                     int B) {
  hipLaunchKernelGGL(k_prologue, dim3(1), dim3(64), 0, s, p, host, ids_src, ids_dst, B);
}

void launch_embed(hipStream_t s, const uint16_t* embed, const int* ids, int vocab, int H, int B, float* X,
                  float* stats, const float* gain, u32x4* a_hi, u32x4* a_lo) {
  hipLaunchKernelGGL(k_embed, dim3(B), dim3(256), 0, s, embed, ids, vocab, H, X, stats, gain, a_hi, a_lo);
}

void launch_fuse(hipStream_t s, const uint16_t* hidden, int n, int S, int H, int D, const float* alpha,
                 const float* gain, float* ustats, u32x4* ua_hi, u32x4* ua_lo, int n_max, int mt_max,
                 StepParams* params, int L) {
  hipLaunchKernelGGL(k_fuse, dim3((H + 511) / 512, n, D), dim3(64), 0, s, hidden, n, S, H, alpha, gain, ustats,
                     ua_hi, ua_lo, n_max, mt_max, params, L);
}

void launch_fused_rows(hipStream_t s, const u32x4* ua_hi, const u32x4* ua_lo, const float* ustats, int n, int H,
                       int D, int n_max, int mt_max, float eps, float* out) {
  hipLaunchKernelGGL(k_fused_rows, dim3(n, D), dim3(256), 0, s, ua_hi, ua_lo, ustats, n, H, D, n_max, mt_max, eps,
                     out);
}

template <int NT, int WAVES>
static void gemm_nw(hipStream_t s, int epi, const GemmArgs& a, dim3 grid) {
  const dim3 block(64 * WAVES);
  switch (epi) {
    case EPI_RESID: hipLaunchKernelGGL((k_gemm<NT, WAVES, EPI_RESID>), grid, block, 0, s, a); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((k_gemm<NT, WAVES, EPI_SWIGLU>), grid, block, 0, s, a); break;
    case EPI_QKV: hipLaunchKernelGGL((k_gemm<NT, WAVES, EPI_QKV>), grid, block, 0, s, a); break;
    case EPI_KVT: hipLaunchKernelGGL((k_gemm<NT, WAVES, EPI_KVT>), grid, block, 0, s, a); break;
    case EPI_ARGMAX: hipLaunchKernelGGL((k_gemm<NT, WAVES, EPI_ARGMAX>), grid, block, 0, s, a); break;
  }
}

bool gemm_shape_supported(int nt_per_block, int waves) {
  return (nt_per_block == 1 && (waves == 8 || waves == 16)) || (nt_per_block == 2 && (waves == 8 || waves == 16)) ||
         (nt_per_block == 4 && (waves == 4 || waves == 8));
}

void launch_gemm(hipStream_t s, int epi, int nt_per_block, int waves, const GemmArgs& a, int layers, int mtiles) {
  const dim3 grid((a.Nt + nt_per_block - 1) / nt_per_block, layers, mtiles);
  if (nt_per_block == 1) {
    if (waves == 16) gemm_nw<1, 16>(s, epi, a, grid);
    else gemm_nw<1, 8>(s, epi, a, grid);
  } else if (nt_per_block == 2) {
    if (waves == 16) gemm_nw<2, 16>(s, epi, a, grid);
    else gemm_nw<2, 8>(s, epi, a, grid);
  } else {
    if (waves == 8) gemm_nw<4, 8>(s, epi, a, grid);
    else gemm_nw<4, 4>(s, epi, a, grid);
  }
}

void launch_argmax_combine(hipStream_t s, const float* pmax, const int* pidx, int groups, int B, int* tokens) {
  hipLaunchKernelGGL(k_argmax_combine, dim3(B), dim3(256), 0, s, pmax, pidx, groups, tokens);
}

template <int HD>
static void attn_hd(hipStream_t s, const AttnArgs& a, int chunk, int n_chunks, bool combine) {
  if (!combine) {
    const dim3 grid(n_chunks, a.n_kv);
    if (chunk == 64) hipLaunchKernelGGL((k_attn<HD, 64>), grid, dim3(512), 0, s, a);
    else hipLaunchKernelGGL((k_attn<HD, 128>), grid, dim3(512), 0, s, a);
  } else {
    const dim3 grid(a.Rpad, a.n_kv);
    if (chunk == 64) hipLaunchKernelGGL((k_attn_combine<HD, 64>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_attn_combine<HD, 128>), grid, dim3(256), 0, s, a);
  }
}

void launch_attention(hipStream_t s, const AttnArgs& a, int hd, int chunk, int n_chunks) {
  if (hd == 64) attn_hd<64>(s, a, chunk, n_chunks, false);
  else attn_hd<128>(s, a, chunk, n_chunks, false);
}

void launch_attn_combine(hipStream_t s, const AttnArgs& a, int hd, int chunk, int n_chunks) {
  if (hd == 64) attn_hd<64>(s, a, chunk, n_chunks, true);
  else attn_hd<128>(s, a, chunk, n_chunks, true);
}

}  // namespace dflare
