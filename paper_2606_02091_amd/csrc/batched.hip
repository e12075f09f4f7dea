// Batched draft step: many sequences share the draft weights, each with its own context
// cache (Sec. 3.2 drafting pass, Eq. 3 and Eq. 4, applied to every sequence).  The
// M = n_seq * B block rows of a call go through the draft layers together, so the
// projections are GEMMs with M up to 1024 rows, bound by the matrix cores rather than by
// the weight stream.
//
// Precision.  GEMM operands are fp16 on the fp16 matrix cores with fp32 accumulation: the
// activations enter as normalised fp16 rows (RMSNorm applied before the GEMM, saturated
// to +-65504), the weights as an fp16 copy of the packed bf16 tiles made once (exact for
// every weight of magnitude in [2^-14, 65504]; smaller ones keep an absolute error below
// 2^-25).  The KV cache is fp16 and attention computes as on the batch-1 path (fp16
// hi/lo queries and probabilities).  One fp16 operand plane does half the matrix-core
// work of the batch-1 path's bf16 hi/lo pair, which matters here because these GEMMs are
// compute bound; its rounding (2^-11 relative) keeps the logits within about 1e-3 of
// the exact values.
#include <math.h>

#include <type_traits>

#include "batched.h"
#include "device_common.h"

namespace dflare {

constexpr int kBT = kBWaves * 64;

// fp16 bits of x, round to nearest even, no saturation (weights)
__device__ __forceinline__ uint32_t f2h_raw(float x) { return __builtin_bit_cast(uint16_t, (_Float16)x); }

// two floats -> packed fp16 pair (saturated), element order low then high
__device__ __forceinline__ uint32_t pack_h2(float a, float b) { return (uint32_t)f2h(a) | ((uint32_t)f2h(b) << 16); }

// 8 bf16 values (one B-operand lane slot) -> 8 fp16 values
__device__ __forceinline__ u32x4 bf16x8_to_f16x8(u32x4 v) {
  u32x4 r;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float lo = __uint_as_float(v[e] << 16), hi = __uint_as_float(v[e] & 0xFFFF0000u);
    r[e] = f2h_raw(lo) | (f2h_raw(hi) << 16);
  }
  return r;
}

// packed bf16 weight tiles -> the same tiles in fp16 (one 16-byte lane slot per thread)
__global__ void k_tiles_to_f16(u32x4* dst, const u32x4* src, long n) {
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x)
    dst[i] = bf16x8_to_f16x8(src[i]);
}

// 8 floats -> one 16-byte fp16 A-fragment slot (saturated)
__device__ __forceinline__ u32x4 pack_h8(const float* v) {
  return u32x4{pack_h2(v[0], v[1]), pack_h2(v[2], v[3]), pack_h2(v[4], v[5]), pack_h2(v[6], v[7])};
}

// deterministic sum over a work-group of 256 threads (fixed shuffle and wave order)
__device__ __forceinline__ float block_sum256(float v, float* red) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) v += __shfl_xor(v, off);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

// f(integral_constant<int, I>) for I = B .. E-1, as straight-line code
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// best (score, id) of 4 rows over the 16 lanes of a quad (ties to the lowest id); lane col 0
// writes them to bv_out[0..3], bi_out[0..3]
__device__ __forceinline__ void row_best_to_lds(float bv[4], int bi[4], int col, float* bv_out, int* bi_out) {
#pragma unroll
  for (int e = 0; e < 4; ++e)
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
      const float ov = __shfl_xor(bv[e], off);
      const int oi = __shfl_xor(bi[e], off);
      if (ov > bv[e] || (ov == bv[e] && oi < bi[e])) {
        bv[e] = ov;
        bi[e] = oi;
      }
    }
  if (col == 0)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      bv_out[e] = bv[e];
      bi_out[e] = bi[e];
    }
}

// ------------------------------------------------------------------------------------------
// GEMM.  Work-group: 4 waves; output tile 128 rows x 64 NW columns (NW = 4, or 3 where the
// narrower tiles fill the CUs better), wave w owning NW 16-column tiles for all 128 rows
// (8 x NW MFMA tiles, 32 NW accumulators per lane); two work-groups share a CU (two waves
// per SIMD), so one wave's MFMAs run while the other waits for LDS or the barrier.  Per
// k-tile (32 deep) a wave reads its NW weight fragments straight from memory (each a coalesced 1 KiB load of its own columns, used
// directly as MFMA operands; the work-groups of the other m-groups of the same columns
// run on the same XCD and meet in its L2) and loads 2 of the 8 A fragments, which go
// through a 2-slot LDS ring so that every wave reads all 8 with one barrier per k-tile.
// The loads of k-tile t + P are issued after the MFMAs of k-tile t; they are never
// skipped (past the last k-tile they repeat it), so the compiler can wait for exactly the
// loads a step needs.
// ------------------------------------------------------------------------------------------
template <int EPI, int NW>
__global__ __launch_bounds__(kBT) __attribute__((amdgpu_waves_per_eu(kBWavesPerSimd, kBWavesPerSimd))) void k_bgemm(
    BGemmArgs g, BRows rows) {
  constexpr int P = kBPrefetch;
  __shared__ u32x4 sa[2][kBM * 64];
  __shared__ int s_slot[kBM * 16];
  __shared__ int s_pos[kBM * 16];
  __shared__ long s_cache[kBM * 16];
  __shared__ float s_bv[kBWaves][kBM * 16];
  __shared__ int s_bi[kBWaves][kBM * 16];
  __shared__ int s_last;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int quad = lane >> 4, col = lane & 15;

  // work-group -> (layer, K part, n-group, m-group).  Work-groups go to the 8 XCDs in
  // turn (id % 8); the m-groups of one (layer, K part, n-group) read the same weight
  // tiles, so they get consecutive ids on one XCD.
  const int Ng = (g.Nt + kBWaves * NW - 1) / (kBWaves * NW), Mg = (g.Mt + kBM - 1) / kBM;
  const int nb = Ng * Mg * g.kg * g.layers;
  const int bid = blockIdx.x;
  const int t = (nb % 8 == 0) ? (bid % 8) * (nb / 8) + bid / 8 : bid;
  const int mg = t % Mg, ng = (t / Mg) % Ng, kz = (t / (Mg * Ng)) % g.kg, layer = t / (Mg * Ng * g.kg);
  const int tile = (layer * Ng + ng) * Mg + mg;
  const int kb = (int)((long)kz * g.Kt / g.kg), ke = (int)((long)(kz + 1) * g.Kt / g.kg);
  const int nk = ke - kb;

  const u32x4* A = g.A + layer * g.a_layer;
  const u32x4* W = g.W + layer * g.w_layer;
  const int nt0 = ng * (kBWaves * NW) + w * NW;
  const u32x4* wp[NW];
#pragma unroll
  for (int n = 0; n < NW; ++n) wp[n] = W + ((long)min(nt0 + n, g.Nt - 1) * g.Kt + kb) * 64 + lane;
  const u32x4* ap[2];
  int astep[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int mt = mg * kBM + 2 * w + j;
    const bool ok = mt < g.Mt;
    ap[j] = ok ? A + ((long)mt * g.Kt + kb) * 64 + lane : g.zero + lane;
    astep[j] = ok ? 64 : 0;
  }
  const int klast = max(nk - 1, 0);

  f32x4 acc[kBM][NW];
#pragma unroll
  for (int m = 0; m < kBM; ++m)
#pragma unroll
    for (int n = 0; n < NW; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto kidx = [&](int i) -> long { return min(i, klast); };
  if (nk > 0) {
    u32x4 wr[P][NW], ar[P][2];
#pragma unroll
    for (int j = 0; j < P; ++j) {
      const long kt = kidx(j);
#pragma unroll
      for (int n = 0; n < NW; ++n) wr[j][n] = wp[n][kt * 64];
      ar[j][0] = ap[0][kt * astep[0]];
      ar[j][1] = ap[1][kt * astep[1]];
    }
    for (int t0 = 0; t0 < nk; t0 += P) {
#pragma unroll
      for (int j = 0; j < P; ++j) {
        const int tk = t0 + j;
        // slot tk % 2 was last read at k-tile tk - 2, before the barrier of k-tile tk - 1
        u32x4* slot = sa[tk & 1];
        slot[(2 * w) * 64 + lane] = ar[j][0];
        slot[(2 * w + 1) * 64 + lane] = ar[j][1];
        __syncthreads();
        if (tk < nk) {
#pragma unroll
          for (int m = 0; m < kBM; ++m) {
            const u32x4 a = slot[m * 64 + lane];
#pragma unroll
            for (int n = 0; n < NW; ++n) acc[m][n] = mfma_h(a, wr[j][n], acc[m][n]);
          }
        }
        const long kt = kidx(tk + P);
#pragma unroll
        for (int n = 0; n < NW; ++n) wr[j][n] = wp[n][kt * 64];
        ar[j][0] = ap[0][kt * astep[0]];
        ar[j][1] = ap[1][kt * astep[1]];
      }
    }
  }

  if (g.kg > 1) {
    // split K: leave this part's tile, then the last part to arrive sums all parts in K order
    // (each 1 KiB block: elements 0-1 of the 64 lanes, then elements 2-3, so that every
    // 8-byte store or load instruction covers 512 contiguous bytes)
    float* mine = g.part + (((long)tile * g.kg + kz) * kBWaves + w) * (kBM * NW * 256);
#pragma unroll
    for (int m = 0; m < kBM; ++m)
#pragma unroll
      for (int n = 0; n < NW; ++n) {
        float* blk = mine + (m * NW + n) * 256;
        const u32x4 v = __builtin_bit_cast(u32x4, acc[m][n]);
        st_wt8(blk + lane * 2, (uint64_t)v[0] | ((uint64_t)v[1] << 32));
        st_wt8(blk + 128 + lane * 2, (uint64_t)v[2] | ((uint64_t)v[3] << 32));
      }
    wait_vm();
    __syncthreads();
    if (tid == 0) {
      const unsigned old = __hip_atomic_fetch_add(g.cnt + tile * 32, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      s_last = old == (unsigned)(g.kg - 1);
    }
    __syncthreads();
    if (!s_last) return;
    if (tid == 0) st_wt(g.cnt + tile * 32, 0u);
    // sum in K-part order, two m-tiles at a time: the 16 loads of one part are issued
    // together, then added
#pragma unroll
    for (int m0 = 0; m0 < kBM; m0 += 2) {
      f32x4 sm[2][NW];
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int n = 0; n < NW; ++n) sm[mi][n] = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int z = 0; z < g.kg; ++z) {
        if (z == kz) {
#pragma unroll
          for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int n = 0; n < NW; ++n) sm[mi][n] += acc[m0 + mi][n];
          continue;
        }
        const float* zb = g.part + (((long)tile * g.kg + z) * kBWaves + w) * (kBM * NW * 256);
        float2 lo[2][NW], hi[2][NW];
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
          for (int n = 0; n < NW; ++n) {
            const float* blk = zb + ((m0 + mi) * NW + n) * 256;
            lo[mi][n] = ld_coh2(blk + lane * 2);
            hi[mi][n] = ld_coh2(blk + 128 + lane * 2);
          }
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
          for (int n = 0; n < NW; ++n) sm[mi][n] += f32x4{lo[mi][n].x, lo[mi][n].y, hi[mi][n].x, hi[mi][n].y};
      }
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int n = 0; n < NW; ++n) acc[m0 + mi][n] = sm[mi][n];
    }
  }

  const int row0 = mg * kBM * 16;
  if constexpr (EPI == BEPI_QKV) {
    // rows -> cache slot and cache base of their sequence
    if (tid < kBM * 16) {
      const int row = min(row0 + tid, g.M - 1);
      int i = 0;
      while (i + 1 < rows.n_seq && row >= rows.off[i + 1]) ++i;
      s_slot[tid] = rows.L[i] + (row - rows.off[i]);
      s_cache[tid] = (long)rows.seq[i] * g.seq_stride + (long)(g.layer0 + layer) * g.cache_layer;
    }
    __syncthreads();
    const int tph = g.hd / 16, half = g.hd / 2;
    const int kvd = g.kv_tiles * 16;
    const float* kvb = g.bias ? g.bias + (long)(g.layer0 + layer) * 2 * kvd : nullptr;
#pragma unroll
    for (int n = 0; n < NW; ++n) {
      const int nt = nt0 + n;
      if (nt >= g.Nt) continue;
      int region, tt;  // 0 = Q, 1 = K, 2 = V
      if (nt < g.q_tiles) {
        region = 0;
        tt = nt;
      } else if (nt < g.q_tiles + g.kv_tiles) {
        region = 1;
        tt = nt - g.q_tiles;
      } else {
        region = 2;
        tt = nt - g.q_tiles - g.kv_tiles;
      }
      const int head = tt / tph, jj = tt % tph;
      const int mm = 8 * jj + (col & 7);
      const int dim = (col < 8) ? mm : half + mm;
      // bias of this lane's column (context K/V only; region 0 has none)
      const float bcol = (kvb && region > 0) ? kvb[(region == 1 ? 0 : kvd) + head * g.hd + (region == 1 ? dim : jj * 16 + col)] : 0.f;
      // the rotary factors of all 32 rows are loaded before any store (rows past M use
      // the slot of row M - 1), so that no load waits behind a store or a branch
      float2 cs[kBM][4];
      if (region < 2) {
#pragma unroll
        for (int m = 0; m < kBM; ++m)
#pragma unroll
          for (int e = 0; e < 4; ++e) cs[m][e] = g.rope[(long)s_slot[m * 16 + quad * 4 + e] * half + mm];
      }
#pragma unroll
      for (int m = 0; m < kBM; ++m) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = m * 16 + quad * 4 + e, row = row0 + r;
          const float x = acc[m][n][e] + bcol;
          const float partner = __shfl_xor(x, 8);
          const int slot = s_slot[r];
          if (region < 2) {
            const float y = (col < 8) ? (x * cs[m][e].x - partner * cs[m][e].y) : (x * cs[m][e].x + partner * cs[m][e].y);
            // query rows past M but inside the Mt m-tiles land in the padding rows of Q,
            // which exist (Q holds Mt * 16 rows or more) and are never read
            if (region == 0) {
              if (mg * kBM + m < g.Mt) g.Q[(long)row * g.q_dim + head * g.hd + dim] = y;
            } else if (row < g.M) {
              g.kc[s_cache[r] + ((long)head * g.Lcap + slot) * g.hd + dim] = f2h(y);
            }
          } else if (row < g.M) {
            g.vt[s_cache[r] + ((long)head * g.hd + jj * 16 + col) * g.Lcap + slot] = f2h(x);
          }
        }
      }
    }
  } else if constexpr (EPI == BEPI_RESID) {
#pragma unroll
    for (int n = 0; n < NW; ++n) {
      const int nt = nt0 + n;
      if (nt >= g.Nt) continue;
      // every row of the m-tiles, those past M included (padding rows of X, never read),
      // so that no load waits behind a branch
      float* xp = g.X + (long)(row0 + quad * 4) * g.H + nt * 16 + col;
      float xv[kBM][4];  // all loads first, then all stores
#pragma unroll
      for (int m = 0; m < kBM; ++m)
#pragma unroll
        for (int e = 0; e < 4; ++e) xv[m][e] = (mg * kBM + m < g.Mt) ? xp[(long)(m * 16 + e) * g.H] : 0.f;
#pragma unroll
      for (int m = 0; m < kBM; ++m)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (mg * kBM + m < g.Mt) xp[(long)(m * 16 + e) * g.H] = xv[m][e] + acc[m][n][e];
    }
  } else if constexpr (EPI == BEPI_SWIGLU) {
    uint32_t* out = reinterpret_cast<uint32_t*>(g.out16);
#pragma unroll
    for (int n = 0; n < NW; ++n) {
      const int nt = nt0 + n;
#pragma unroll
      for (int m = 0; m < kBM; ++m)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int row = row0 + m * 16 + quad * 4 + e;
          const float gt = acc[m][n][e];
          const float up = __shfl_xor(gt, 8);
          const float hv = (col < 8) ? gt / (1.0f + expf(-gt)) * up : 0.f;
          const float h1 = __shfl_xor(hv, 1);
          if (nt < g.Nt && row < g.M && col < 8 && (col & 1) == 0)
            out[frag_off(row, nt * 8 + col, g.out_kt) >> 1] = pack_h2(hv, h1);
        }
    }
  } else if constexpr (EPI == BEPI_BIAS16) {
    uint32_t* out = reinterpret_cast<uint32_t*>(g.out16);
#pragma unroll
    for (int n = 0; n < NW; ++n) {
      const int nt = nt0 + n;
      const float bcol = (g.bias && nt < g.Nt) ? g.bias[nt * 16 + col] : 0.f;
#pragma unroll
      for (int m = 0; m < kBM; ++m)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int row = row0 + m * 16 + quad * 4 + e;
          const float y = acc[m][n][e] + bcol;
          const float y1 = __shfl_xor(y, 1);
          if (nt < g.Nt && row < g.M && (col & 1) == 0) out[frag_off(row, nt * 16 + col, g.out_kt) >> 1] = pack_h2(y, y1);
        }
    }
  } else if constexpr (EPI == BEPI_ARGMAX) {
    // best (score, id) of each row over this wave's 64 columns, then over the 4 waves;
    // ties go to the lowest id (ids grow with n and col)
    if (!(g.inv_temp > 0.f)) {
#pragma unroll
      for (int m = 0; m < kBM; ++m) {
        float bv[4];
        int bi[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          bv[e] = -INFINITY;
          bi[e] = 0x7FFFFFFF;
        }
#pragma unroll
        for (int n = 0; n < NW; ++n) {
          const int vc = (nt0 + n) * 16 + col;
          const bool ok = vc < g.V;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int row = row0 + m * 16 + quad * 4 + e;
            const float z = acc[m][n][e];
            if (ok && row < g.M && g.logits) g.logits[(long)row * g.V + vc] = z;
            if (ok && (z > bv[e] || (z == bv[e] && vc < bi[e]))) {
              bv[e] = z;
              bi[e] = vc;
            }
          }
        }
        row_best_to_lds(bv, bi, col, s_bv[w] + m * 16 + quad * 4, s_bi[w] + m * 16 + quad * 4);
      }
    } else {
      // sampling: score z / T + Gumbel noise of the row's (sequence slot, block position).
      // The noise costs a Philox call per four positions, so this part runs as rolled loops
      // (one copy of the generator in the code): per m-tile the thread's 16 scaled logits go
      // to its own LDS slots (the A ring, idle after the k loop), the noise is added there,
      // and the best is taken from there.
      if (tid < kBM * 16) {
        const int row = min(row0 + tid, g.M - 1);
        int i = 0;
        while (i + 1 < rows.n_seq && row >= rows.off[i + 1]) ++i;
        s_slot[tid] = rows.seq[i];
        s_pos[tid] = row - rows.off[i];
      }
      __syncthreads();  // also: every wave is past its last read of the A ring
      uint64_t words[4];
      float* zs = reinterpret_cast<float*>(&sa[0][0]) + tid;  // [16][kBT], this thread's column
      // m is unrolled at compile time (the accumulators are indexed by constants) while the
      // noise loop inside stays rolled
      static_for<0, kBM>([&](auto mc) {
        constexpr int m = decltype(mc)::value;
#pragma unroll
        for (int n = 0; n < NW; ++n) {
          const int vc = (nt0 + n) * 16 + col;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int row = row0 + m * 16 + quad * 4 + e;
            const float z = acc[m][n][e];
            if (vc < g.V && row < g.M && g.logits) g.logits[(long)row * g.V + vc] = z;
            zs[(n * 4 + e) * kBT] = z * g.inv_temp;
          }
        }
        const int r0 = m * 16 + quad * 4;
        // rows 4 q .. 4 q + 3 of one sequence share one Philox call, else one call per row
        const bool grouped = (s_pos[r0] & 3) == 0 && s_pos[r0 + 3] == s_pos[r0] + 3 && s_slot[r0 + 3] == s_slot[r0];
#pragma unroll 1
        for (int j = 0; j < NW * 4; ++j) {
          const int n = j >> 2, e = j & 3;
          if (e == 0 || !grouped) {
            const int pos = s_pos[r0 + e], slot = s_slot[r0 + e];
            gumbel_words(g.seed, (nt0 + n) * 16 + col, pos >> 2, g.draw, slot, words);
          }
          const int k = grouped ? e : (s_pos[r0 + e] & 3);
          zs[j * kBT] += gumbel_of_word(k == 0 ? words[0] : k == 1 ? words[1] : k == 2 ? words[2] : words[3]);
        }
        float bv[4];
        int bi[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          bv[e] = -INFINITY;
          bi[e] = 0x7FFFFFFF;
        }
#pragma unroll
        for (int n = 0; n < NW; ++n) {
          const int vc = (nt0 + n) * 16 + col;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float v = zs[(n * 4 + e) * kBT];
            if (vc < g.V && (v > bv[e] || (v == bv[e] && vc < bi[e]))) {
              bv[e] = v;
              bi[e] = vc;
            }
          }
        }
        row_best_to_lds(bv, bi, col, s_bv[w] + r0, s_bi[w] + r0);
      });
    }
    __syncthreads();
    if (tid < kBM * 16) {
      float v = s_bv[0][tid];
      int ix = s_bi[0][tid];
#pragma unroll
      for (int q = 1; q < kBWaves; ++q) {
        const float ov = s_bv[q][tid];
        const int oi = s_bi[q][tid];
        if (ov > v || (ov == v && oi < ix)) {
          v = ov;
          ix = oi;
        }
      }
      const int row = row0 + tid;
      if (row < g.Mt * 16) {
        g.pmax[(long)ng * g.pld + row] = v;
        g.pidx[(long)ng * g.pld + row] = ix;
      }
    }
  }
}

// best over the LM head's n-groups, per row (one wave per row)
__global__ __launch_bounds__(64) void k_bargmax(const float* pmax, const int* pidx, int ngroups, int pld, int M,
                                                int* tokens) {
  const int row = blockIdx.x, lane = threadIdx.x;
  if (row >= M) return;
  float v = -INFINITY;
  int ix = 0x7FFFFFFF;
  for (int n = lane; n < ngroups; n += 64) {
    const float ov = pmax[(long)n * pld + row];
    const int oi = pidx[(long)n * pld + row];
    if (ov > v || (ov == v && oi < ix)) {
      v = ov;
      ix = oi;
    }
  }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const float ov = __shfl_xor(v, off);
    const int oi = __shfl_xor(ix, off);
    if (ov > v || (ov == v && oi < ix)) {
      v = ov;
      ix = oi;
    }
  }
  if (lane == 0) tokens[row] = (ix == 0x7FFFFFFF) ? 0 : ix;
}


// RMSNorm of row blockIdx.x of X [M, H] (fp32) with gain g into fp16 A fragments.  One
// work-group of 256 threads per row, 8 consecutive columns per thread and step.
__global__ __launch_bounds__(256) void k_bnorm(const float* X, int H, const float* gain, float eps, u32x4* A,
                                               int a_kt) {
  __shared__ float red[4];
  const int row = blockIdx.x;
  const float* x = X + (long)row * H;
  float sq = 0.f;
  for (int k0 = threadIdx.x * 8; k0 < H; k0 += 2048) {
    const f32x4 a = *reinterpret_cast<const f32x4*>(x + k0), b = *reinterpret_cast<const f32x4*>(x + k0 + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) sq += a[e] * a[e] + b[e] * b[e];
  }
  const float rstd = rsqrtf(block_sum256(sq, red) / H + eps);
  for (int k0 = threadIdx.x * 8; k0 < H; k0 += 2048) {
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = x[k0 + e] * rstd * gain[k0 + e];
    A[frag_off(row, k0, a_kt) >> 3] = pack_h8(v);
  }
}

// embedding rows X = E[ids] (ids clamped into [0, V)), then as k_bnorm
__global__ __launch_bounds__(256) void k_bembed_norm(const uint16_t* embed, const int32_t* ids, int H, int V,
                                                     const float* gain, float eps, float* X, u32x4* A, int a_kt) {
  __shared__ float red[4];
  const int row = blockIdx.x;
  int id = ids[row];
  id = id < 0 ? 0 : (id >= V ? V - 1 : id);
  const uint16_t* er = embed + (long)id * H;
  float* x = X + (long)row * H;
  float sq = 0.f;
  for (int k0 = threadIdx.x * 8; k0 < H; k0 += 2048) {
    const u32x4 u = *reinterpret_cast<const u32x4*>(er + k0);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float a = bf2f(u[e] & 0xFFFFu), b = bf2f(u[e] >> 16);
      x[k0 + 2 * e] = a;
      x[k0 + 2 * e + 1] = b;
      sq += a * a + b * b;
    }
  }
  const float rstd = rsqrtf(block_sum256(sq, red) / H + eps);
  for (int k0 = threadIdx.x * 8; k0 < H; k0 += 2048) {
    const u32x4 u = *reinterpret_cast<const u32x4*>(er + k0);
    float v[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[2 * e] = bf2f(u[e] & 0xFFFFu) * rstd * gain[k0 + 2 * e];
      v[2 * e + 1] = bf2f(u[e] >> 16) * rstd * gain[k0 + 2 * e + 1];
    }
    A[frag_off(row, k0, a_kt) >> 3] = pack_h8(v);
  }
}

// layer fusion (Eq. 3) of appended row r for draft layer i: u = sum_j alpha[i, j] h^(j)[r]
// in j order, then f = RMSNorm(u; g_fuse^(i)) into the fp16 A fragments of layer i.  One
// work-group per (row, layer); the S target rows of r are read from HBM once and found in
// L2 by the work-groups of the other layers.
__global__ __launch_bounds__(256) void k_bfuse(const uint16_t* hidden, int ld, int S, int H, const float* alpha,
                                               const float* gain, float eps, u32x4* A, int mt_max) {
  constexpr int kMaxChunks = 4;  // H <= 8192
  __shared__ float red[4];
  const int r = blockIdx.x, i = blockIdx.y;
  const int Kt = H / 32;
  float u[kMaxChunks][8];
  float sq = 0.f;
#pragma unroll
  for (int c = 0; c < kMaxChunks; ++c) {
    const int k0 = threadIdx.x * 8 + c * 2048;
#pragma unroll
    for (int e = 0; e < 8; ++e) u[c][e] = 0.f;
    if (k0 < H) {
      // 12 target rows in flight per step, summed in j order
      for (int j0 = 0; j0 < S; j0 += 12) {
        u32x4 v[12];
#pragma unroll
        for (int jj = 0; jj < 12; ++jj)
          v[jj] = *reinterpret_cast<const u32x4*>(hidden + ((long)min(j0 + jj, S - 1) * ld + r) * H + k0);
#pragma unroll
        for (int jj = 0; jj < 12; ++jj) {
          if (j0 + jj < S) {
            const float a = alpha[i * S + j0 + jj];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              u[c][2 * e] = fmaf(a, bf2f(v[jj][e] & 0xFFFFu), u[c][2 * e]);
              u[c][2 * e + 1] = fmaf(a, bf2f(v[jj][e] >> 16), u[c][2 * e + 1]);
            }
          }
        }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) sq += u[c][e] * u[c][e];
    }
  }
  const float rstd = rsqrtf(block_sum256(sq, red) / H + eps);
  u32x4* Ai = A + (long)i * mt_max * Kt * 64;
#pragma unroll
  for (int c = 0; c < kMaxChunks; ++c) {
    const int k0 = threadIdx.x * 8 + c * 2048;
    if (k0 < H) {
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = u[c][e] * rstd * gain[(long)i * H + k0 + e];
      Ai[frag_off(r, k0, Kt) >> 3] = pack_h8(v);
    }
  }
}

// The same fusion for all D <= 8 layers of appended row r in one work-group of 512 threads
// (H <= 4096, 8 columns per thread): the S target rows of r are read once and each value
// feeds the D weighted sums, so HBM sees the rows once however the work-groups are placed.
// The sums are formed in the same order as k_bfuse forms them for one layer; the RMS
// statistics over the 8 waves.
constexpr int kBFuseMaxD = 8;
__global__ __launch_bounds__(512) void k_bfuse_all(const uint16_t* hidden, int ld, int S, int H, int D,
                                                   const float* alpha, const float* gain, float eps, u32x4* A,
                                                   int mt_max) {
  constexpr int JB = 12;  // target rows in flight
  __shared__ float red[kBFuseMaxD][8];
  const int r = blockIdx.x;
  const int Kt = H / 32;
  const bool has = threadIdx.x * 8 < H;
  const int k0 = has ? threadIdx.x * 8 : 0;
  float u[kBFuseMaxD][8];
#pragma unroll
  for (int i = 0; i < kBFuseMaxD; ++i)
#pragma unroll
    for (int e = 0; e < 8; ++e) u[i][e] = 0.f;
  for (int j0 = 0; j0 < S; j0 += JB) {
    u32x4 v[JB];
#pragma unroll
    for (int jj = 0; jj < JB; ++jj)
      v[jj] = *reinterpret_cast<const u32x4*>(hidden + ((long)min(j0 + jj, S - 1) * ld + r) * H + k0);
#pragma unroll
    for (int jj = 0; jj < JB; ++jj) {
      if (j0 + jj < S) {
#pragma unroll
        for (int i = 0; i < kBFuseMaxD; ++i) {
          if (i < D) {
            const float a = alpha[i * S + j0 + jj];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              u[i][2 * e] = fmaf(a, bf2f(v[jj][e] & 0xFFFFu), u[i][2 * e]);
              u[i][2 * e + 1] = fmaf(a, bf2f(v[jj][e] >> 16), u[i][2 * e + 1]);
            }
          }
        }
      }
    }
  }
  float sq[kBFuseMaxD];
#pragma unroll
  for (int i = 0; i < kBFuseMaxD; ++i) {
    sq[i] = 0.f;
    if (has)
#pragma unroll
      for (int e = 0; e < 8; ++e) sq[i] += u[i][e] * u[i][e];
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) sq[i] += __shfl_xor(sq[i], off);
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0)
#pragma unroll
    for (int i = 0; i < kBFuseMaxD; ++i) red[i][w] = sq[i];
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kBFuseMaxD; ++i) {
    if (i >= D) break;
    const float tot = ((red[i][0] + red[i][1]) + (red[i][2] + red[i][3])) + ((red[i][4] + red[i][5]) + (red[i][6] + red[i][7]));
    const float rstd = rsqrtf(tot / H + eps);
    if (has) {
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = u[i][e] * rstd * gain[(long)i * H + k0 + e];
      u32x4* Ai = A + (long)i * mt_max * Kt * 64;
      Ai[frag_off(r, k0, Kt) >> 3] = pack_h8(v);
    }
  }
}

// debug: fp16 A fragments of D layers -> rows [D, n, H] fp32
__global__ void k_bfrag_rows(const u32x4* A, int n, int H, int mt_max, float* out) {
  const int r = blockIdx.x, i = blockIdx.y, Kt = H / 32;
  const uint16_t* a = reinterpret_cast<const uint16_t*>(A + (long)i * mt_max * Kt * 64);
  for (int k = threadIdx.x; k < H; k += blockDim.x) out[((long)i * n + r) * H + k] = h2f(a[frag_off(r, k, Kt)]);
}

// DFlash FC input (Eq. 1): row r of the call, the S target rows of its position side by
// side in layer order, as fp16 A fragments [mt][S*H/32][64]; block (row r, target layer j),
// a thread converts 8 consecutive values (one 16-byte fragment slot).
__global__ __launch_bounds__(256) void k_bfrag_cat(const uint16_t* hidden, int ld, int S, int H, u32x4* A) {
  const int r = blockIdx.x, j = blockIdx.y, Kt = S * H / 32;
  for (int k0 = threadIdx.x * 8; k0 < H; k0 += 256 * 8) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(hidden + ((long)j * ld + r) * H + k0);
    float f[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[2 * e] = bf2f(v[e] & 0xFFFFu);
      f[2 * e + 1] = bf2f(v[e] >> 16);
    }
    A[frag_off(r, j * H + k0, Kt) >> 3] = pack_h8(f);
  }
}

// ------------------------------------------------------------------------------------------
// attention over ragged contexts (Sec. 3.2: no mask; the block rows of a sequence see its
// whole context and the whole block, whose keys and values are already in the cache at
// slots L .. L + B - 1).  Work item (sequence i, key range r, KV head g): keys
// r * kBKeys .. min((r + 1) * kBKeys, L + B) - 1 in blocks of 64, against the G * B query
// rows of head g (query tile qt = 16 rows, row r' = head offset * B + block row).  The
// 4 waves share each key block, staged in LDS (K rows and V^T rows, fp16, with XOR-
// swizzled 16-byte pieces) while the next block is loaded into registers; each wave
// keeps its query tiles' running max, sum and output in registers (online softmax, log2
// domain).  Scores are formed transposed (S^T = K Q^T) so that the probabilities are
// the B operand of the P V product; queries and probabilities enter as fp16 hi/lo pairs.
// ------------------------------------------------------------------------------------------
template <int HD, int TPW, int KB, int NBUF>
__global__ __launch_bounds__(256, 2) void k_battn(BAttnArgs a, BRows rows) {
  // KB keys per block; NBUF LDS buffers (2: the next block is stored while this one is
  // computed; 1: stored after it, behind a second barrier)
  constexpr int KC = HD / 8, VC = KB / 8;  // 16-byte pieces per K row / per V^T row
  constexpr int KP = KB * KC, VP = HD * VC;
  constexpr int NT = 256, PER = (KP + VP) / NT;
  static_assert(KP % NT == 0 && VP % NT == 0, "pieces split evenly");
  __shared__ u32x4 st[NBUF][KP + VP];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int q = lane & 15, quad = lane >> 4;

  const int j = blockIdx.x;
  int i = 0;
  while (i + 1 < rows.n_seq && j >= rows.ipfx[i + 1]) ++i;
  const int L = rows.L[i];
  const int rr = (j - rows.ipfx[i]) / a.n_kv, g = (j - rows.ipfx[i]) % a.n_kv;
  const int kbeg = rr * kBKeys, kend = min(kbeg + kBKeys, L + a.B);
  const int nblk = (kend - kbeg + KB - 1) / KB;
  const long cache = (long)rows.seq[i] * a.seq_stride + (long)a.layer * a.cache_layer;
  const uint16_t* kc = a.kc + cache + (long)g * a.Lcap * HD;
  const uint16_t* vt = a.vt + cache + (long)g * HD * a.Lcap;
  const int G = a.n_q / a.n_kv, R = G * a.B, QT = (R + 15) / 16;

  // loads of key block b into registers.  Every lane loads (pieces past kend repeat the
  // last key row or the last 8-key group), so that no load sits in a branch; those pieces
  // are zeroed when they are stored to LDS.  The cache is read once per step: nontemporal
  // loads (115 -> 107 us per layer at 32 sequences).
  // blocks loaded ahead of the one being computed: two, or one where the query tiles of a
  // wave already fill the registers (set b % PF holds block b)
  constexpr int PF = (NBUF == 1 || (HD == 128 && TPW == 2)) ? 1 : 2;
  u32x4 pcs[PF][PER];
  auto fetch = [&](int b, u32x4* dst) {
    const int k0 = kbeg + b * KB;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int p = k * NT + tid;  // the K / V^T split is static per k (KP is a multiple of NT)
      if (k * NT < KP) {
        const int r = p / KC, c = p % KC;
        dst[k] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kc + (long)min(k0 + r, kend - 1) * HD + c * 8));
      } else {
        const int pv = p - KP, d = pv / VC, c = pv % VC;
        dst[k] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vt + (long)d * a.Lcap + min(k0 + c * 8, (kend - 1) & ~7)));
      }
    }
  };
  auto stash = [&](int b, int buf, const u32x4* src) {
    const int k0 = kbeg + b * KB;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int p = k * NT + tid;
      if (k * NT < KP) {
        const int r = p / KC, c = p % KC;
        const bool ok = k0 + r < kend;
        const u32x4 v = src[k];
        st[buf][r * KC + (c ^ (r & 7))] = u32x4{ok ? v[0] : 0u, ok ? v[1] : 0u, ok ? v[2] : 0u, ok ? v[3] : 0u};
      } else {
        const int pv = p - KP, d = pv / VC, c = pv % VC;
        const u32x4 v = src[k];
        const int nv = kend - (k0 + c * 8);  // keys of this 8-key group before kend
        u32x4 z;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t lo = (2 * e < nv) ? 0xFFFFu : 0u, hi = (2 * e + 1 < nv) ? 0xFFFF0000u : 0u;
          z[e] = v[e] & (lo | hi);
        }
        // rows with bit 3 of d set hold the piece's two 8-byte halves swapped, so that the 16
        // lanes of one read (16 dim rows, one half each) reach 16 different bank pairs
        if (d & 8) z = u32x4{z[2], z[3], z[0], z[1]};
        st[buf][KP + d * VC + (c ^ (d & 7))] = z;
      }
    }
  };

  // this wave's query tiles: hi/lo fp16 fragments of Q^T (scaled), running statistics
  u32x4 qh[TPW][HD / 32], ql[TPW][HD / 32];
  f32x4 o[TPW][HD / 16];
  float m_run[TPW], l_run[TPW];
  const int q_dim = a.n_q * HD;
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    const int r = (w + 4 * t) * 16 + q;
    const bool rv = r < R;
    const int bb = rv ? r % a.B : 0, h = g * G + (rv ? r / a.B : 0);
    const float* src = a.Q + (long)(rows.off[i] + bb) * q_dim + h * HD;
    const float sc = rv ? a.qscale : 0.f;  // rows past R: a valid row, scaled to zero
#pragma unroll
    for (int ks = 0; ks < HD / 32; ++ks) {
      const f32x4 x0 = *reinterpret_cast<const f32x4*>(src + ks * 32 + quad * 8);
      const f32x4 x1 = *reinterpret_cast<const f32x4*>(src + ks * 32 + quad * 8 + 4);
      float v[8] = {x0[0] * sc, x0[1] * sc, x0[2] * sc, x0[3] * sc, x1[0] * sc, x1[1] * sc, x1[2] * sc, x1[3] * sc};
      split_pack8_h(v, qh[t][ks], ql[t][ks]);
    }
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) o[t][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    m_run[t] = -INFINITY;
    l_run[t] = 0.f;
  }

  fetch(0, pcs[0]);
  if (PF == 2 && nblk > 1) fetch(1, pcs[PF - 1]);
  stash(0, 0, pcs[0]);
  __syncthreads();
  const char* base0 = reinterpret_cast<const char*>(&st[0][0]);
  const int vx = (quad >> 1);
  // block b: the loads of block b + PF go out, block b is computed from LDS, block b + 1
  // goes to the other LDS buffer, which was last read in block b - 1
  auto step = [&](int b, u32x4* ahead, const u32x4* nxt1) {
    if (b + PF < nblk) fetch(b + PF, ahead);
    const char* lds = base0 + (NBUF == 2 ? (b & 1) : 0) * (KP + VP) * 16;
    const int k0 = kbeg + b * KB;
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
      if (w + 4 * t >= QT) continue;
      // scores S^T for 4 key tiles of 16
      f32x4 sc[KB / 16];
#pragma unroll
      for (int kt = 0; kt < KB / 16; ++kt) {
        f32x4 hacc = {0.f, 0.f, 0.f, 0.f}, lacc = hacc;
        const int row = kt * 16 + q;
#pragma unroll
        for (int ks = 0; ks < HD / 32; ++ks) {
          const u32x4 kv = *reinterpret_cast<const u32x4*>(lds + (row * KC + ((ks * 4 + quad) ^ (row & 7))) * 16);
          hacc = mfma_h(kv, qh[t][ks], hacc);
          lacc = mfma_h(kv, ql[t][ks], lacc);
        }
        sc[kt] = hacc + lacc;
      }
      if (k0 + KB > kend) {  // the block reaches past the item's last key
#pragma unroll
        for (int kt = 0; kt < KB / 16; ++kt)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (k0 + kt * 16 + quad * 4 + e >= kend) sc[kt][e] = -INFINITY;
      }
      float mb = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < KB / 16; ++kt)
#pragma unroll
        for (int e = 0; e < 4; ++e) mb = fmaxf(mb, sc[kt][e]);
      mb = fmaxf(mb, __shfl_xor(mb, 16));
      mb = fmaxf(mb, __shfl_xor(mb, 32));
      // the running maximum moves only when the block's maximum exceeds it by more than 8 (so
      // the unnormalised probabilities stay below 2^8); the rescale of the output and the sum
      // then runs for the whole wave, with factor 1 on rows that did not move
      const bool grow = mb > m_run[t] + 8.f;
      if (__builtin_amdgcn_ballot_w64(grow) != 0) {
        const float mn = grow ? mb : m_run[t];
        const float scale = __builtin_amdgcn_exp2f(m_run[t] - mn);
        l_run[t] *= scale;
#pragma unroll
        for (int dt = 0; dt < HD / 16; ++dt) o[t][dt] *= scale;
        m_run[t] = mn;
      }
      float ls = 0.f;
#pragma unroll
      for (int kt = 0; kt < KB / 16; ++kt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p = __builtin_amdgcn_exp2f(sc[kt][e] - m_run[t]);
          sc[kt][e] = p;
          ls += p;
        }
      ls += __shfl_xor(ls, 16);
      ls += __shfl_xor(ls, 32);
      l_run[t] += ls;
      // O^T += V^T P^T, 32 keys per step
#pragma unroll
      for (int kk = 0; kk < KB / 32; ++kk) {
        float pv[8] = {sc[2 * kk][0], sc[2 * kk][1], sc[2 * kk][2], sc[2 * kk][3],
                       sc[2 * kk + 1][0], sc[2 * kk + 1][1], sc[2 * kk + 1][2], sc[2 * kk + 1][3]};
        u32x4 ph, pl;
        split_pack8_hz(pv, ph, pl);
#pragma unroll
        for (int dt = 0; dt < HD / 16; ++dt) {
          const int d = dt * 16 + q;
          const int p0 = (4 * kk + vx) ^ (d & 7), p1 = (4 * kk + 2 + vx) ^ (d & 7);
          const char* vrow = lds + (KP + d * VC) * 16 + (((quad & 1) ^ ((d >> 3) & 1)) * 8);
          const u32x2 x0 = *reinterpret_cast<const u32x2*>(vrow + p0 * 16);
          const u32x2 x1 = *reinterpret_cast<const u32x2*>(vrow + p1 * 16);
          const u32x4 vv = {x0[0], x0[1], x1[0], x1[1]};
          o[t][dt] = mfma_h(vv, ph, o[t][dt]);
          o[t][dt] = mfma_h(vv, pl, o[t][dt]);
        }
      }
    }
    if (b + 1 < nblk) {
      if (NBUF == 1) __syncthreads();  // every wave is done with the buffer
      stash(b + 1, NBUF == 2 ? (b + 1) & 1 : 0, nxt1);
      __syncthreads();
    }
  };
  for (int b = 0; b < nblk; b += 2) {
    step(b, pcs[0], pcs[PF - 1]);
    if (b + 1 < nblk) step(b + 1, pcs[PF - 1], pcs[0]);
  }

#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    const int r = (w + 4 * t) * 16 + q;
    if (w + 4 * t < QT && r < R) {
      const long base = (long)j * a.Rpad + r;
#pragma unroll
      for (int dt = 0; dt < HD / 16; ++dt)
        *reinterpret_cast<f32x4*>(a.OP + base * HD + dt * 16 + quad * 4) = o[t][dt];
      if (quad == 0) a.ML[base] = make_float2(m_run[t], l_run[t]);
    }
  }
}

// merge the key-range partials of query row r of head g of sequence i (one wave per row)
// and write the fp16 A fragments of the output projection at row off[i] + r % B
template <int HD>
__global__ __launch_bounds__(64) void k_bcomb(BAttnArgs a, BRows rows, u32x4* out16, int a_kt) {
  constexpr int DPL = HD / 64;
  const int lane = threadIdx.x;
  const int G = a.n_q / a.n_kv, R = G * a.B;
  const int it = blockIdx.x;
  const int i = it / (a.n_kv * R), g = (it / R) % a.n_kv, r = it % R;
  if (i >= rows.n_seq) return;
  const int nr = (rows.L[i] + a.B + kBKeys - 1) / kBKeys;
  const long jb = rows.ipfx[i] + g;  // item of range 0; range c at jb + c * n_kv
  float M = -INFINITY;
  for (int c = lane; c < nr; c += 64) M = fmaxf(M, a.ML[(jb + (long)c * a.n_kv) * a.Rpad + r].x);
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) M = fmaxf(M, __shfl_xor(M, off));
  float num[DPL], den = 0.f;
#pragma unroll
  for (int e = 0; e < DPL; ++e) num[e] = 0.f;
  for (int c = 0; c < nr; ++c) {
    const long base = (jb + (long)c * a.n_kv) * a.Rpad + r;
    const float2 mc = a.ML[base];
    const float wgt = exp2f(mc.x - M);
    den += wgt * mc.y;
#pragma unroll
    for (int e = 0; e < DPL; ++e) num[e] += wgt * a.OP[base * HD + lane * DPL + e];
  }
  const float inv = 1.0f / den;
  const int row = rows.off[i] + r % a.B, h = g * G + r / a.B;
  uint32_t* o = reinterpret_cast<uint32_t*>(out16);
  if constexpr (DPL == 2) {
    o[frag_off(row, h * HD + 2 * lane, a_kt) >> 1] = pack_h2(num[0] * inv, num[1] * inv);
  } else {
    const float y = num[0] * inv, y1 = __shfl_xor(y, 1);
    if ((lane & 1) == 0) o[frag_off(row, h * HD + lane, a_kt) >> 1] = pack_h2(y, y1);
  }
}

// ------------------------------------------------------------------------------------------
// launchers
// ------------------------------------------------------------------------------------------
int bgemm_groups(int Nt, int Mt, int nw) {
  const int bn = kBWaves * nw;
  return ((Nt + bn - 1) / bn) * ((Mt + kBM - 1) / kBM);
}

void launch_tiles_to_f16(hipStream_t s, u32x4* dst, const u32x4* src, long n) {
  hipLaunchKernelGGL(k_tiles_to_f16, dim3(2048), dim3(256), 0, s, dst, src, n);
}

void launch_bgemm(hipStream_t s, int epi, const BGemmArgs& g, const BRows& rows) {
  const dim3 grid(bgemm_groups(g.Nt, g.Mt, g.nw) * g.kg * g.layers);
  switch (epi) {
    case BEPI_QKV:
      if (g.nw == 3) hipLaunchKernelGGL((k_bgemm<BEPI_QKV, 3>), grid, dim3(kBT), 0, s, g, rows);
      else hipLaunchKernelGGL((k_bgemm<BEPI_QKV, kBNW>), grid, dim3(kBT), 0, s, g, rows);
      break;
    case BEPI_RESID:
      if (g.nw == 3) hipLaunchKernelGGL((k_bgemm<BEPI_RESID, 3>), grid, dim3(kBT), 0, s, g, rows);
      else hipLaunchKernelGGL((k_bgemm<BEPI_RESID, kBNW>), grid, dim3(kBT), 0, s, g, rows);
      break;
    case BEPI_SWIGLU:
      if (g.nw == 3) hipLaunchKernelGGL((k_bgemm<BEPI_SWIGLU, 3>), grid, dim3(kBT), 0, s, g, rows);
      else hipLaunchKernelGGL((k_bgemm<BEPI_SWIGLU, kBNW>), grid, dim3(kBT), 0, s, g, rows);
      break;
    case BEPI_BIAS16: hipLaunchKernelGGL((k_bgemm<BEPI_BIAS16, kBNW>), grid, dim3(kBT), 0, s, g, rows); break;
    default: hipLaunchKernelGGL((k_bgemm<BEPI_ARGMAX, kBNW>), grid, dim3(kBT), 0, s, g, rows); break;
  }
}

void launch_bargmax(hipStream_t s, const float* pmax, const int* pidx, int ngroups, int pld, int M, int* tokens) {
  hipLaunchKernelGGL(k_bargmax, dim3(M), dim3(64), 0, s, pmax, pidx, ngroups, pld, M, tokens);
}

void launch_bnorm(hipStream_t s, const float* X, int M, int H, const float* gain, float eps, u32x4* A, int a_kt) {
  hipLaunchKernelGGL(k_bnorm, dim3(M), dim3(256), 0, s, X, H, gain, eps, A, a_kt);
}

void launch_bembed_norm(hipStream_t s, const uint16_t* embed, const int32_t* ids, int M, int H, int V,
                        const float* gain, float eps, float* X, u32x4* A, int a_kt) {
  hipLaunchKernelGGL(k_bembed_norm, dim3(M), dim3(256), 0, s, embed, ids, H, V, gain, eps, X, A, a_kt);
}

void launch_bfuse(hipStream_t s, const uint16_t* hidden, int N, int ld, int S, int H, int D, const float* alpha,
                  const float* gain, float eps, u32x4* A, int mt_max) {
  if (D <= kBFuseMaxD && H <= 4096)
    hipLaunchKernelGGL(k_bfuse_all, dim3(N), dim3(512), 0, s, hidden, ld, S, H, D, alpha, gain, eps, A, mt_max);
  else
    hipLaunchKernelGGL(k_bfuse, dim3(N, D), dim3(256), 0, s, hidden, ld, S, H, alpha, gain, eps, A, mt_max);
}

void launch_bfrag_cat(hipStream_t s, const uint16_t* hidden, int N, int ld, int S, int H, u32x4* A) {
  hipLaunchKernelGGL(k_bfrag_cat, dim3(N, S), dim3(256), 0, s, hidden, ld, S, H, A);
}

void launch_bfrag_rows(hipStream_t s, const u32x4* A, int n, int H, int D, int mt_max, float* out) {
  hipLaunchKernelGGL(k_bfrag_rows, dim3(n, D), dim3(256), 0, s, A, n, H, mt_max, out);
}

template <int KB, int NBUF>
static void launch_battn_v(hipStream_t s, int hd, const BAttnArgs& a, const BRows& rows, int items) {
  const bool two = (a.n_q / a.n_kv) * a.B > 64;  // more than 4 query tiles: two per wave
  if (hd == 64) {
    if (two) hipLaunchKernelGGL((k_battn<64, 2, KB, NBUF>), dim3(items), dim3(256), 0, s, a, rows);
    else hipLaunchKernelGGL((k_battn<64, 1, KB, NBUF>), dim3(items), dim3(256), 0, s, a, rows);
  } else {
    if (two) hipLaunchKernelGGL((k_battn<128, 2, KB, NBUF>), dim3(items), dim3(256), 0, s, a, rows);
    else hipLaunchKernelGGL((k_battn<128, 1, KB, NBUF>), dim3(items), dim3(256), 0, s, a, rows);
  }
}

void launch_battn(hipStream_t s, int hd, const BAttnArgs& a, const BRows& rows, int items) {
  launch_battn_v<64, 2>(s, hd, a, rows, items);
}

void launch_bcomb(hipStream_t s, int hd, const BAttnArgs& a, const BRows& rows, u32x4* out16, int a_kt) {
  const int R = (a.n_q / a.n_kv) * a.B;
  const dim3 grid(rows.n_seq * a.n_kv * R);
  if (hd == 64) hipLaunchKernelGGL(k_bcomb<64>, grid, dim3(64), 0, s, a, rows, out16, a_kt);
  else hipLaunchKernelGGL(k_bcomb<128>, grid, dim3(64), 0, s, a, rows, out16, a_kt);
}

}  // namespace dflare
