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
// embedding gather: X[b, :] = E[id_b, :] (fp32) and per-16-column sums of squares
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_embed(const uint16_t* __restrict__ E, const int* __restrict__ ids,
                                               int vocab, int H, float* X, float* stats) {
  const int b = blockIdx.x;
  int id = ids[b];
  id = id < 0 ? 0 : (id >= vocab ? vocab - 1 : id);
  const uint16_t* row = E + (long)id * H;
  for (int k0 = threadIdx.x * 8; k0 < H; k0 += blockDim.x * 8) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(row + k0);
    float f[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[2 * e] = bf2f(v[e] & 0xFFFFu);
      f[2 * e + 1] = bf2f(v[e] >> 16);
    }
    float sq = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) sq += f[e] * f[e];
    float* xo = X + (long)b * H + k0;
    *reinterpret_cast<float4*>(xo) = make_float4(f[0], f[1], f[2], f[3]);
    *reinterpret_cast<float4*>(xo + 4) = make_float4(f[4], f[5], f[6], f[7]);
    sq += __shfl_xor(sq, 1);
    if ((threadIdx.x & 1) == 0) stats[(long)b * (H / 16) + k0 / 16] = sq;
  }
}

// ------------------------------------------------------------------------------------------
// layer fusion (Eq. 3): u^(i)[r, k] = sum_j alpha[i, j] h^(j)[r, k] for all D draft layers from
// one read of the S target rows; the RMS statistics are kept as per-16-column partial sums.
// grid (ceil(H / 512), n), block 64, LDS S * 1 KiB.
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(64) void k_fuse(const uint16_t* __restrict__ hidden, int n, int S, int H, int D,
                                             const float* __restrict__ alpha, float* U, float* ustats,
                                             int n_max) {
  extern __shared__ u32x4 sh[];
  const int lane = threadIdx.x;
  const int r = blockIdx.y;
  const int k0 = blockIdx.x * 512 + lane * 8;
  const bool ok = k0 < H;
  for (int j = 0; j < S; ++j) {
    u32x4 v = {0u, 0u, 0u, 0u};
    if (ok) v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(hidden + ((long)j * n + r) * H + k0));
    sh[j * 64 + lane] = v;
  }
  // each lane reads back only its own slots: no barrier needed
  for (int i = 0; i < D; ++i) {
    float u[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < S; ++j) {
      const float a = alpha[i * S + j];
      const u32x4 v = sh[j * 64 + lane];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        u[2 * e] = fmaf(a, bf2f(v[e] & 0xFFFFu), u[2 * e]);
        u[2 * e + 1] = fmaf(a, bf2f(v[e] >> 16), u[2 * e + 1]);
      }
    }
    float sq = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) sq += u[e] * u[e];
    sq += __shfl_xor(sq, 1);
    if (ok) {
      float* o = U + ((long)i * n_max + r) * H + k0;
      *reinterpret_cast<float4*>(o) = make_float4(u[0], u[1], u[2], u[3]);
      *reinterpret_cast<float4*>(o + 4) = make_float4(u[4], u[5], u[6], u[7]);
      if ((lane & 1) == 0) ustats[((long)i * n_max + r) * (H / 16) + k0 / 16] = sq;
    }
  }
}

// debug: materialise f^(i) = u * rstd * g (fp32), [D, n, H]
__global__ void k_fused_rows(const float* U, const float* ustats, const float* gain, int n, int H, int D,
                             int n_max, float eps, float* out) {
  const int r = blockIdx.x, i = blockIdx.y;
  __shared__ float s_r;
  if (threadIdx.x == 0) {
    float s = 0.f;
    for (int t = 0; t < H / 16; ++t) s += ustats[((long)i * n_max + r) * (H / 16) + t];
    s_r = rsqrtf(s / H + eps);
  }
  __syncthreads();
  for (int k = threadIdx.x; k < H; k += blockDim.x)
    out[((long)i * n + r) * H + k] = U[((long)i * n_max + r) * H + k] * s_r * gain[(long)i * H + k];
}

// ------------------------------------------------------------------------------------------
// weight-streaming GEMM, y[M<=16 per m-tile, N] = x[M, K] W^T, split-K over blocks.
// Block = 4 waves; block (group, split) owns n-tiles [group*4*NT, +4*NT) and k-tiles
// [split*kt_per_split, +kt_per_split).  Activations of the k range are normalised (optional
// RMSNorm from partial statistics), split into bf16 hi/lo and staged in LDS in A-operand
// order; each wave streams its NT weight tiles.  The last block of a group to arrive sums
// the split partials in fixed order (deterministic) and runs the fused epilogue.
// ------------------------------------------------------------------------------------------
template <int NT, int EPI>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs a) {
  constexpr int U = (8 / NT) < 2 ? 2 : (8 / NT);
  extern __shared__ u32x4 lds[];
  __shared__ float s_rstd[16];
  __shared__ int s_last;
  __shared__ float s_bv[4][16];
  __shared__ int s_bi[4][16];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int quad = lane >> 4, col = lane & 15;
  const int groups = (a.Nt + 4 * NT - 1) / (4 * NT);
  const int group = blockIdx.x % groups, split = blockIdx.x / groups;
  const int layer = blockIdx.y, mt = blockIdx.z;
  const int kt0 = split * a.kt_per_split;
  const int kt1 = min(a.Kt, kt0 + a.kt_per_split);
  const int nk = kt1 - kt0;
  const int M = (EPI == EPI_KVT) ? a.e.params->n_new : a.M;
  if (mt * 16 >= M) return;  // whole m-tile idle: every split of it leaves together

  // 1. per-row 1/rms from the producer's partial sums of squares
  if (a.stats) {
    const int row = tid >> 4, part = tid & 15;
    float s = 0.f;
    if (mt * 16 + row < M) {
      const float* st = a.stats + layer * a.stats_layer_stride + (long)(mt * 16 + row) * a.n_stat;
      for (int t = part; t < a.n_stat; t += 16) s += st[t];
    }
    s += __shfl_xor(s, 8);
    s += __shfl_xor(s, 4);
    s += __shfl_xor(s, 2);
    s += __shfl_xor(s, 1);
    if (part == 0) s_rstd[row] = rsqrtf(s * a.inv_dim + a.eps);
  }
  __syncthreads();

  // 2. stage the activation slice as bf16 hi/lo A fragments
  u32x4* lhi = lds;
  u32x4* llo = lds + a.kt_per_split * 64;
  {
    const float* X = a.X + layer * a.x_layer_stride;
    const float* G = a.gain ? a.gain + layer * a.gain_layer_stride : nullptr;
    for (int idx = tid; idx < nk * 64; idx += 256) {
      const int t = idx >> 6, l = idx & 63, r = l & 15;
      const int row = mt * 16 + r;
      const int k = (kt0 + t) * 32 + (l >> 4) * 8;
      float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      if (row < M) {
        const float4 x0 = *reinterpret_cast<const float4*>(X + (long)row * a.ldx + k);
        const float4 x1 = *reinterpret_cast<const float4*>(X + (long)row * a.ldx + k + 4);
        v[0] = x0.x; v[1] = x0.y; v[2] = x0.z; v[3] = x0.w;
        v[4] = x1.x; v[5] = x1.y; v[6] = x1.z; v[7] = x1.w;
        const float sc = a.stats ? s_rstd[r] : 1.0f;
        if (G) {
          const float4 g0 = *reinterpret_cast<const float4*>(G + k);
          const float4 g1 = *reinterpret_cast<const float4*>(G + k + 4);
          v[0] *= sc * g0.x; v[1] *= sc * g0.y; v[2] *= sc * g0.z; v[3] *= sc * g0.w;
          v[4] *= sc * g1.x; v[5] *= sc * g1.y; v[6] *= sc * g1.z; v[7] *= sc * g1.w;
        } else if (a.stats) {
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] *= sc;
        }
      }
      u32x4 hi, lo;
      split_pack8(v, hi, lo);
      lhi[idx] = hi;
      llo[idx] = lo;
    }
  }
  __syncthreads();

  // 3. stream the weight tiles through the matrix cores
  const int nt_base = group * 4 * NT + wave * NT;
  f32x4 acc[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const u32x4* Wl = a.W + layer * a.w_layer_stride;
  for (int t = 0; t < nk; t += U) {
    u32x4 b[U][NT];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        const int nt = nt_base + j;
        b[u][j] = u32x4{0u, 0u, 0u, 0u};
        if (t + u < nk && nt < a.Nt)
          b[u][j] = __builtin_nontemporal_load(Wl + ((long)nt * a.Kt + kt0 + t + u) * 64 + lane);
      }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (t + u < nk) {
        const u32x4 ah = lhi[(t + u) * 64 + lane];
        const u32x4 al = llo[(t + u) * 64 + lane];
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          acc[j] = mfma(ah, b[u][j], acc[j]);
          acc[j] = mfma(al, b[u][j], acc[j]);
        }
      }
    }
  }

  // 4. split-K: last arriving block sums the partials in split order
  if (a.splits > 1) {
    const long ptile = (long)(layer * gridDim.z + mt) * a.splits;  // (layer, m-tile) slab
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const int nt = nt_base + j;
      if (nt < a.Nt)
        *reinterpret_cast<f32x4*>(a.partials + (((ptile + split) * a.Nt + nt) * 64 + lane) * 4) = acc[j];
    }
    __threadfence();
    __syncthreads();
    if (tid == 0) {
      unsigned* c = a.counters + (long)(layer * gridDim.z + mt) * groups + group;
      const unsigned prev = atomicAdd(c, 1u);
      s_last = (prev == (unsigned)(a.splits - 1));
      if (s_last) *c = 0u;  // every split has arrived: reset for the next launch
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const int nt = nt_base + j;
      f32x4 s = {0.f, 0.f, 0.f, 0.f};
      if (nt < a.Nt)
        for (int sp = 0; sp < a.splits; ++sp)
          s += *reinterpret_cast<const f32x4*>(a.partials + (((ptile + sp) * a.Nt + nt) * 64 + lane) * 4);
      acc[j] = s;
    }
  }

  // 5. epilogues.  Lane holds rows mt*16 + 4*quad + i (i < 4) of output column nt*16 + col.
  const EpiArgs& e = a.e;
  if constexpr (EPI == EPI_RESID) {
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const int nt = nt_base + j;
      if (nt >= a.Nt) continue;  // wave-uniform
      float sq[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = mt * 16 + quad * 4 + i;
        float x = 0.f;
        if (row < M) {
          float* p = e.out + (long)row * e.ldo + nt * 16 + col;
          x = *p + acc[j][i];
          *p = x;
        }
        sq[i] = x * x;
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
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const int nt = nt_base + j;
      if (nt >= a.Nt) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float v = acc[j][i];
        const float up = __shfl_xor(v, 8);
        const int row = mt * 16 + quad * 4 + i;
        if (col < 8 && row < M) e.out[(long)row * e.ldo + nt * 8 + col] = v / (1.0f + expf(-v)) * up;
      }
    }
  } else if constexpr (EPI == EPI_QKV || EPI == EPI_KVT) {
    const int L = e.params->L;
    const int tph = e.hd / 16, half = e.hd / 2;
    uint16_t* kc = e.kc + (EPI == EPI_KVT ? layer * e.cache_layer_stride : 0);
    uint16_t* vt = e.vt + (EPI == EPI_KVT ? layer * e.cache_layer_stride : 0);
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const int nt = nt_base + j;
      if (nt >= a.Nt) continue;
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
        const float v = acc[j][i];
        const float partner = __shfl_xor(v, 8);
        if (region < 2) {
          const int m = 8 * jj + (col & 7);
          const int dim = (col < 8) ? m : half + m;
          const float2 cs = e.rope[(long)pos * half + m];
          const float y = (col < 8) ? (v * cs.x - partner * cs.y) : (v * cs.x + partner * cs.y);
          if (valid) {
            if (region == 0)
              e.out[(long)row * e.ldo + head * e.hd + dim] = y;
            else
              kc[((long)head * e.Lcap + slot) * e.hd + dim] = (uint16_t)f2bf(y);
          }
        } else if (valid) {
          const int dim = jj * 16 + col;
          vt[((long)head * e.hd + dim) * e.Lcap + slot] = (uint16_t)f2bf(v);
        }
      }
    }
  } else if constexpr (EPI == EPI_ARGMAX) {
    float bv[4];
    int bi[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) { bv[i] = -INFINITY; bi[i] = 0x7FFFFFFF; }
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const int nt = nt_base + j;
      const int c = nt * 16 + col;
      const bool ok = nt < a.Nt && c < e.vocab;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = quad * 4 + i;
        const float v = acc[j][i];
        if (ok && e.logits && row < e.B) e.logits[(long)row * e.vocab + c] = v;
        if (ok && (v > bv[i] || (v == bv[i] && c < bi[i]))) { bv[i] = v; bi[i] = c; }
      }
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
    __syncthreads();
    if (tid < 16) {
      float v = s_bv[0][tid];
      int ix = s_bi[0][tid];
      for (int w = 1; w < 4; ++w) {
        const float ov = s_bv[w][tid];
        const int oi = s_bi[w][tid];
        if (ov > v || (ov == v && oi < ix)) { v = ov; ix = oi; }
      }
      e.pmax[(long)tid * groups + group] = v;
      e.pidx[(long)tid * groups + group] = ix;
    }
    __threadfence();
    __syncthreads();
    if (tid == 0) {
      const unsigned prev = atomicAdd(e.counter2, 1u);
      s_last = (prev == (unsigned)(groups - 1));
      if (s_last) *e.counter2 = 0u;
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    // final combine: 16 threads per row
    const int row = tid >> 4, part = tid & 15;
    float v = -INFINITY;
    int ix = 0x7FFFFFFF;
    for (int g = part; g < groups; g += 16) {
      const float ov = e.pmax[(long)row * groups + g];
      const int oi = e.pidx[(long)row * groups + g];
      if (ov > v || (ov == v && oi < ix)) { v = ov; ix = oi; }
    }
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
      const float ov = __shfl_xor(v, off);
      const int oi = __shfl_xor(ix, off);
      if (ov > v || (ov == v && oi < ix)) { v = ov; ix = oi; }
    }
    if (part == 0 && row < e.B) e.tokens[row] = (ix == 0x7FFFFFFF) ? 0 : ix;
  }
}

// ------------------------------------------------------------------------------------------
// block attention, split over the key axis (Sec. 3.2: no mask, every block row sees the
// whole context and the whole block).  Block (chunk c, KV head g); wave w takes 16 query rows
// r = w*16 + lane%16 of the G*B rows that share head g (r -> query head g*G + r/B, block
// position r%B).  Scores are formed transposed, S^T = K Q^T, so that the probabilities land
// in exactly the B-operand layout of the P V product and never leave registers.
// ------------------------------------------------------------------------------------------
template <int HD, int CK>
__global__ __launch_bounds__(512) void k_attn(AttnArgs a) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int quad = lane >> 4, q = lane & 15;
  const int g = blockIdx.y, c = blockIdx.x;
  const int Lk = a.params->L + a.B;
  const int kbeg = c * CK;
  if (kbeg >= Lk) return;
  const int kend = min(Lk, kbeg + CK);
  const int nkeys = kend - kbeg;
  const int G = a.n_q / a.n_kv;
  const int R = G * a.B;
  const int r = w * 16 + q;
  const bool rv = r < R;
  const int b = rv ? r % a.B : 0;
  const int h = g * G + (rv ? r / a.B : 0);

  u32x4 qh[HD / 32], ql[HD / 32];
#pragma unroll
  for (int ks = 0; ks < HD / 32; ++ks) {
    float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (rv) {
      const float* src = a.Q + (long)b * a.q_dim + h * HD + ks * 32 + quad * 8;
      const float4 x0 = *reinterpret_cast<const float4*>(src);
      const float4 x1 = *reinterpret_cast<const float4*>(src + 4);
      v[0] = x0.x * a.qscale; v[1] = x0.y * a.qscale; v[2] = x0.z * a.qscale; v[3] = x0.w * a.qscale;
      v[4] = x1.x * a.qscale; v[5] = x1.y * a.qscale; v[6] = x1.z * a.qscale; v[7] = x1.w * a.qscale;
    }
    split_pack8(v, qh[ks], ql[ks]);
  }

  const uint16_t* Kg = a.kc + (long)g * a.Lcap * HD;
  f32x4 s[CK / 16];
#pragma unroll
  for (int kt = 0; kt < CK / 16; ++kt) {
    const int key = kbeg + kt * 16 + q;
    u32x4 kv[HD / 32];
#pragma unroll
    for (int ks = 0; ks < HD / 32; ++ks) {
      kv[ks] = u32x4{0u, 0u, 0u, 0u};
      if (key < kend) kv[ks] = *reinterpret_cast<const u32x4*>(Kg + (long)key * HD + ks * 32 + quad * 8);
    }
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < HD / 32; ++ks) {
      acc = mfma(kv[ks], qh[ks], acc);
      acc = mfma(kv[ks], ql[ks], acc);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (kt * 16 + quad * 4 + i >= nkeys) acc[i] = -INFINITY;
    s[kt] = acc;
  }
  // softmax statistics per query row (column q), in the log2 domain
  float m = -INFINITY;
#pragma unroll
  for (int kt = 0; kt < CK / 16; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i) m = fmaxf(m, s[kt][i]);
  m = fmaxf(m, __shfl_xor(m, 16));
  m = fmaxf(m, __shfl_xor(m, 32));
  float l = 0.f;
#pragma unroll
  for (int kt = 0; kt < CK / 16; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float p = exp2f(s[kt][i] - m);
      s[kt][i] = p;
      l += p;
    }
  l += __shfl_xor(l, 16);
  l += __shfl_xor(l, 32);

  // O^T = V^T P^T over the chunk
  const uint16_t* Vg = a.vt + (long)g * HD * a.Lcap;
  f32x4 o[HD / 16];
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kk = 0; kk < CK / 32; ++kk) {
    float pv[8] = {s[2 * kk][0], s[2 * kk][1], s[2 * kk][2], s[2 * kk][3],
                   s[2 * kk + 1][0], s[2 * kk + 1][1], s[2 * kk + 1][2], s[2 * kk + 1][3]};
    u32x4 ph, pl;
    split_pack8(pv, ph, pl);
    const int k0 = kbeg + kk * 32 + quad * 4;  // keys k0..k0+3 and k0+16..k0+19
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) {
      const uint16_t* vp = Vg + (long)(dt * 16 + q) * a.Lcap;
      u32x2 v0 = {0u, 0u}, v1 = {0u, 0u};
      if (k0 < kend) v0 = *reinterpret_cast<const u32x2*>(vp + k0);
      if (k0 + 16 < kend) v1 = *reinterpret_cast<const u32x2*>(vp + k0 + 16);
      // zero values of keys past the end (their p is 0, but stale memory may hold non-finite bits)
      if (k0 + 4 > kend) {
        const int nv = kend - k0;
        if (nv <= 0) v0 = u32x2{0u, 0u};
        else {
          if (nv < 2) v0[0] &= 0xFFFFu;
          if (nv < 3) v0[1] = 0u;
          if (nv < 4) v0[1] &= 0xFFFFu;
        }
      }
      if (k0 + 20 > kend) {
        const int nv = kend - (k0 + 16);
        if (nv <= 0) v1 = u32x2{0u, 0u};
        else {
          if (nv < 2) v1[0] &= 0xFFFFu;
          if (nv < 3) v1[1] = 0u;
          if (nv < 4) v1[1] &= 0xFFFFu;
        }
      }
      const u32x4 av = {v0[0], v0[1], v1[0], v1[1]};
      o[dt] = mfma(av, ph, o[dt]);
      o[dt] = mfma(av, pl, o[dt]);
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

// combine the chunk partials: O = sum_c 2^(m_c - M) O_c / sum_c 2^(m_c - M) l_c
template <int HD, int CK>
__global__ __launch_bounds__(256) void k_attn_combine(AttnArgs a) {
  const int g = blockIdx.y;
  const int idx = blockIdx.x * 256 + threadIdx.x;
  const int r = idx / HD, d = idx % HD;
  const int G = a.n_q / a.n_kv;
  const int R = G * a.B;
  if (r >= R) return;
  const int nch = (a.params->L + a.B + CK - 1) / CK;
  float M = -INFINITY;
  for (int c = 0; c < nch; ++c) M = fmaxf(M, a.ml[((long)c * a.n_kv + g) * a.Rpad + r].x);
  float num = 0.f, den = 0.f;
  for (int c = 0; c < nch; ++c) {
    const long base = ((long)c * a.n_kv + g) * a.Rpad + r;
    const float2 ml = a.ml[base];
    const float wgt = exp2f(ml.x - M);
    den += wgt * ml.y;
    num += wgt * a.opart[base * HD + d];
  }
  const int b = r % a.B, h = g * G + r / a.B;
  a.out[(long)b * a.q_dim + h * HD + d] = num / den;
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
                  float* stats) {
  hipLaunchKernelGGL(k_embed, dim3(B), dim3(256), 0, s, embed, ids, vocab, H, X, stats);
}

void launch_fuse(hipStream_t s, const uint16_t* hidden, int n, int S, int H, int D, const float* alpha, float* U,
                 float* ustats, int n_max) {
  hipLaunchKernelGGL(k_fuse, dim3((H + 511) / 512, n), dim3(64), (size_t)S * 1024, s, hidden, n, S, H, D, alpha,
                     U, ustats, n_max);
}

void launch_fused_rows(hipStream_t s, const float* U, const float* ustats, const float* gain, int n, int H, int D,
                       int n_max, float eps, float* out) {
  hipLaunchKernelGGL(k_fused_rows, dim3(n, D), dim3(256), 0, s, U, ustats, gain, n, H, D, n_max, eps, out);
}

size_t gemm_lds_bytes(int kt_per_split) { return (size_t)kt_per_split * 64 * 16 * 2; }

template <int NT>
static void gemm_nt(hipStream_t s, int epi, const GemmArgs& a, dim3 grid, size_t lds) {
  switch (epi) {
    case EPI_RESID: hipLaunchKernelGGL((k_gemm<NT, EPI_RESID>), grid, dim3(256), lds, s, a); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((k_gemm<NT, EPI_SWIGLU>), grid, dim3(256), lds, s, a); break;
    case EPI_QKV: hipLaunchKernelGGL((k_gemm<NT, EPI_QKV>), grid, dim3(256), lds, s, a); break;
    case EPI_KVT: hipLaunchKernelGGL((k_gemm<NT, EPI_KVT>), grid, dim3(256), lds, s, a); break;
    case EPI_ARGMAX: hipLaunchKernelGGL((k_gemm<NT, EPI_ARGMAX>), grid, dim3(256), lds, s, a); break;
  }
}

void launch_gemm(hipStream_t s, int epi, int nt_per_wave, const GemmArgs& a, int layers, int mtiles) {
  const int groups = (a.Nt + 4 * nt_per_wave - 1) / (4 * nt_per_wave);
  const dim3 grid(groups * a.splits, layers, mtiles);
  const size_t lds = gemm_lds_bytes(a.kt_per_split);
  switch (nt_per_wave) {
    case 1: gemm_nt<1>(s, epi, a, grid, lds); break;
    case 2: gemm_nt<2>(s, epi, a, grid, lds); break;
    case 4: gemm_nt<4>(s, epi, a, grid, lds); break;
  }
}

template <int HD>
static void attn_hd(hipStream_t s, const AttnArgs& a, int chunk, int n_chunks, bool combine) {
  const int threads = a.Rpad / 16 * 64;
  if (!combine) {
    const dim3 grid(n_chunks, a.n_kv);
    switch (chunk) {
      case 64: hipLaunchKernelGGL((k_attn<HD, 64>), grid, dim3(threads), 0, s, a); break;
      case 128: hipLaunchKernelGGL((k_attn<HD, 128>), grid, dim3(threads), 0, s, a); break;
      case 256: hipLaunchKernelGGL((k_attn<HD, 256>), grid, dim3(threads), 0, s, a); break;
    }
  } else {
    const dim3 grid((a.Rpad * HD + 255) / 256, a.n_kv);
    switch (chunk) {
      case 64: hipLaunchKernelGGL((k_attn_combine<HD, 64>), grid, dim3(256), 0, s, a); break;
      case 128: hipLaunchKernelGGL((k_attn_combine<HD, 128>), grid, dim3(256), 0, s, a); break;
      case 256: hipLaunchKernelGGL((k_attn_combine<HD, 256>), grid, dim3(256), 0, s, a); break;
    }
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
