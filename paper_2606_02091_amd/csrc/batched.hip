// Batched draft step: many sequences share the draft weights, each with its own context
// cache (Sec. 3.2 drafting pass, Eq. 3 and Eq. 4, applied to every sequence).  The
// M = n_seq * B block rows of a call go through the draft layers together, so the
// projections are real GEMMs: tiles of 128 x 128 outputs staged through LDS on the matrix
// cores, optionally split over K into fp32 slices, followed by an epilogue kernel per
// operator (RoPE and cache store, residual and norm statistics, SwiGLU, argmax).  Numerics
// match the batch-1 path: bf16 weights against hi/lo bf16 activations, fp32 accumulation,
// fp16 KV cache, fp16 hi/lo queries and probabilities in attention.
#include <math.h>

#include "batched.h"
#include "device_common.h"

namespace dflare {

constexpr int kBT = 512;  // GEMM work-group: 8 waves
constexpr int kBK = 2;    // k-tiles per LDS stage
constexpr int kBF = 2 * kBM * kBK + kBN * kBK;  // fragments per stage: A hi/lo, then W
static_assert(kBF % 8 == 0, "fragments split evenly over the waves");

// ------------------------------------------------------------------------------------------
// GEMM: Y = A W^T for A given as hi/lo bf16 fragments [mt][a_kt][64] and W packed
// [nt][Kt][64].  Work-group (n-group ng, m-group mg, K part kz): 8 m-tiles x 8 n-tiles of
// output over k-tiles [kb, ke).  Wave w computes m-tiles 2 (w & 3) + {0, 1} against n-tiles
// 4 (w >> 2) + {0 .. 3}.  Stages of kBK k-tiles are copied global -> registers -> LDS
// (double buffered, one barrier per stage); every fragment is a contiguous 1 KiB block read
// back by lane l at l * 16 bytes, so LDS accesses are conflict-free.  A fragments of
// m-tiles >= Mt or k-tiles >= ke read a zero fragment; W tiles past the matrix are clamped
// (their outputs are dropped).
// ------------------------------------------------------------------------------------------
template <bool ARGMAX>
__global__ __launch_bounds__(kBT) void k_bgemm(BGemmArgs g) {
  __shared__ u32x4 st[2][kBF * 64];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = w & 3, wn = w >> 2;
  // Work-groups are dispatched to the 8 XCDs in turn (id % 8).  The m-groups of one
  // (n-group, K part) read the same weight tiles, so they are given consecutive ids
  // on one XCD and meet in its L2.
  const int Ng = (g.Nt + kBN - 1) / kBN, Mg = (g.Mt + kBM - 1) / kBM;
  const int nb = Ng * Mg * g.kg;
  const int bid = blockIdx.x;
  const int t = (nb % 8 == 0) ? (bid % 8) * (nb / 8) + bid / 8 : bid;
  const int mg = t % Mg, ng = (t / Mg) % Ng, kz = t / (Mg * Ng);
  const int kb = (int)((long)kz * g.Kt / g.kg), ke = (int)((long)(kz + 1) * g.Kt / g.kg);
  const int nst = (ke - kb + kBK - 1) / kBK;

  // fragment f of a stage: f < 2*kBM*kBK: A (k = f / (2 kBM), m = (f / 2) % kBM, plane f % 2);
  // else W (k = (f - A) / kBN, n = (f - A) % kBN).  Wave w copies fragments w, w + 8, ...
  constexpr int FA = 2 * kBM * kBK, PERW = kBF / 8;
  auto src = [&](int f, int s) -> const u32x4* {
    if (f < FA) {
      const int k = f / (2 * kBM), m = (f / 2) % kBM, pl = f & 1;
      const int mt = mg * kBM + m, kt = kb + s * kBK + k;
      if (mt >= g.Mt || kt >= ke) return g.zero + lane;
      return (pl ? g.Alo : g.Ahi) + ((long)mt * g.a_kt + kt) * 64 + lane;
    }
    const int f2 = f - FA, k = f2 / kBN, n = f2 % kBN;
    const int nt = min(ng * kBN + n, g.Nt - 1), kt = min(kb + s * kBK + k, g.Kt - 1);
    return g.W + ((long)nt * g.Kt + kt) * 64 + lane;
  };
  u32x4 ld[PERW];
  auto fetch = [&](int s) {
#pragma unroll
    for (int i = 0; i < PERW; ++i) ld[i] = *src(w + 8 * i, s);
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int i = 0; i < PERW; ++i) st[buf][(w + 8 * i) * 64 + lane] = ld[i];
  };

  f32x4 acc[2][4];
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (nst > 0) {
    fetch(0);
    stash(0);
    __syncthreads();
    if (nst > 1) fetch(1);
  }
  for (int s = 0; s < nst; ++s) {
    const u32x4* sb = st[s & 1];
#pragma unroll
    for (int k = 0; k < kBK; ++k) {
      u32x4 ah[2], al[2], wv[4];
#pragma unroll
      for (int mi = 0; mi < 2; ++mi) {
        const int m = 2 * wm + mi;
        ah[mi] = sb[(k * 2 * kBM + 2 * m) * 64 + lane];
        al[mi] = sb[(k * 2 * kBM + 2 * m + 1) * 64 + lane];
      }
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) wv[ni] = sb[(FA + k * kBN + 4 * wn + ni) * 64 + lane];
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) {
          acc[mi][ni] = mfma(ah[mi], wv[ni], acc[mi][ni]);
          acc[mi][ni] = mfma(al[mi], wv[ni], acc[mi][ni]);
        }
    }
    if (s + 1 < nst) {
      stash((s + 1) & 1);  // this buffer was last read in stage s - 1, before the barrier below
      __syncthreads();
      if (s + 2 < nst) fetch(s + 2);
    }
  }

  const int quad = lane >> 4, col = lane & 15;
  if constexpr (!ARGMAX) {
    float* Y = g.Y + (long)kz * g.Mt * 16 * g.ldy;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) {
        const int mt = mg * kBM + 2 * wm + mi, nt = ng * kBN + 4 * wn + ni;
        if (mt < g.Mt && nt < g.Nt)
#pragma unroll
          for (int i = 0; i < 4; ++i) Y[(long)(mt * 16 + quad * 4 + i) * g.ldy + nt * 16 + col] = acc[mi][ni][i];
      }
  } else {
    // LM head: logits scaled by the final RMSNorm's 1/rms; best (logit, id) per row of this
    // n-group, ties to the lowest id (tiles visited in id order)
    __syncthreads();  // the stage buffers are reused below
    float* sv = reinterpret_cast<float*>(&st[0][0]);   // [2 wn][kBM * 16 rows]
    int* si = reinterpret_cast<int*>(sv + 2 * kBM * 16);
#pragma unroll
    for (int mi = 0; mi < 2; ++mi) {
      const int mt = mg * kBM + 2 * wm + mi;
      float bv[4];
      int bi[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        bv[i] = -INFINITY;
        bi[i] = 0x7FFFFFFF;
      }
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) {
        const int nt = ng * kBN + 4 * wn + ni;
        const int vc = nt * 16 + col;
        const bool ok = nt < g.Nt && vc < g.V;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = mt * 16 + quad * 4 + i;
          const float v = acc[mi][ni][i] * (mt < g.Mt ? g.rstd[row] : 0.f);
          if (ok && row < g.M && g.logits) g.logits[(long)row * g.V + vc] = v;
          if (ok && (v > bv[i] || (v == bv[i] && vc < bi[i]))) {
            bv[i] = v;
            bi[i] = vc;
          }
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) {
          const float ov = __shfl_xor(bv[i], off);
          const int oi = __shfl_xor(bi[i], off);
          if (ov > bv[i] || (ov == bv[i] && oi < bi[i])) {
            bv[i] = ov;
            bi[i] = oi;
          }
        }
      if (col == 0)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = (2 * wm + mi) * 16 + quad * 4 + i;
          sv[wn * kBM * 16 + r] = bv[i];
          si[wn * kBM * 16 + r] = bi[i];
        }
    }
    __syncthreads();
    if (tid < kBM * 16) {
      const int row = mg * kBM * 16 + tid;
      float v = sv[tid];
      int ix = si[tid];
      const float v1 = sv[kBM * 16 + tid];
      const int i1 = si[kBM * 16 + tid];
      if (v1 > v || (v1 == v && i1 < ix)) {
        v = v1;
        ix = i1;
      }
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

// 1/rms of each row from its per-16-column sums of squares [rows][n_st] (one wave per row)
__global__ __launch_bounds__(64) void k_brstd(const float* stats, int n_st, int M, float inv_dim, float eps,
                                              float* rstd) {
  const int row = blockIdx.x, lane = threadIdx.x;
  if (row >= M) return;
  float s = 0.f;
  for (int t = lane; t < n_st; t += 64) s += stats[(long)row * n_st + t];
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) s += __shfl_xor(s, off);
  if (lane == 0) rstd[row] = rsqrtf(s * inv_dim + eps);
}

// the 16 outputs of (row, columns c0 .. c0+15): sum of the K slices, in slice order
__device__ __forceinline__ void bsum16(const BEpiArgs& e, int row, int c0, float* v) {
#pragma unroll
  for (int c = 0; c < 16; ++c) v[c] = 0.f;
  for (int z = 0; z < e.kg; ++z) {
    const f32x4* p = reinterpret_cast<const f32x4*>(e.Y + ((long)z * e.Mpad + row) * e.ldy + c0);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const f32x4 x = p[j];
#pragma unroll
      for (int i = 0; i < 4; ++i) v[4 * j + i] += x[i];
    }
  }
}

// A fragments of 8 consecutive columns k0 .. k0+7 of `row` (k0 a multiple of 8)
__device__ __forceinline__ void store_frag8(u32x4* hi, u32x4* lo, int row, int k0, int a_kt, const float* v) {
  u32x4 h, l;
  split_pack8(v, h, l);
  const long o = frag_off(row, k0, a_kt) >> 3;
  hi[o] = h;
  lo[o] = l;
}

// ---- epilogues: one thread per (row, 16-column output tile) ----
// EMBED: X = E[ids]; stats; A fragments of x * g
__global__ void k_bembed(const uint16_t* embed, const int32_t* ids, int M, int H, int V, const float* gain,
                         float* X, float* stats, u32x4* ahi, u32x4* alo, int a_kt) {
  const int n_st = H / 16;
  const long item = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (item >= (long)M * n_st) return;
  const int row = (int)(item / n_st), t = (int)(item % n_st);
  int id = ids[row];
  id = id < 0 ? 0 : (id >= V ? V - 1 : id);
  float x[16], sq = 0.f;
  const u32x4* e = reinterpret_cast<const u32x4*>(embed + (long)id * H + t * 16);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const u32x4 v = e[h];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[h * 8 + 2 * j] = bf2f(v[j] & 0xFFFFu);
      x[h * 8 + 2 * j + 1] = bf2f(v[j] >> 16);
    }
  }
  float y[16];
#pragma unroll
  for (int c = 0; c < 16; ++c) {
    X[(long)row * H + t * 16 + c] = x[c];
    sq += x[c] * x[c];
    y[c] = x[c] * gain[t * 16 + c];
  }
  stats[(long)row * n_st + t] = sq;
  store_frag8(ahi, alo, row, t * 16, a_kt, y);
  store_frag8(ahi, alo, row, t * 16 + 8, a_kt, y + 8);
}

// RESID: X += y (slices summed); stats of the new rows; A fragments of x * g_next
__global__ void k_bresid(BEpiArgs e) {
  const int n_st = e.H / 16;
  const long item = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (item >= (long)e.M * n_st) return;
  const int row = (int)(item / n_st), t = (int)(item % n_st);
  float x[16], y[16], sq = 0.f;
  bsum16(e, row, t * 16, x);
  f32x4* px = reinterpret_cast<f32x4*>(e.X + (long)row * e.H + t * 16);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    f32x4 v = px[j];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[i] += x[4 * j + i];
      x[4 * j + i] = v[i];
    }
    px[j] = v;
  }
#pragma unroll
  for (int c = 0; c < 16; ++c) {
    sq += x[c] * x[c];
    y[c] = x[c] * e.gain[t * 16 + c];
  }
  e.stats[(long)row * n_st + t] = sq;
  store_frag8(e.ahi, e.alo, row, t * 16, e.a_kt, y);
  store_frag8(e.ahi, e.alo, row, t * 16 + 8, e.a_kt, y + 8);
}

// SWIGLU: packed tile t holds gate rows 8t .. 8t+7 then the matching up rows
__global__ void k_bswiglu(BEpiArgs e) {
  const int nt = e.N / 16;
  const long item = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (item >= (long)e.M * nt) return;
  const int row = (int)(item / nt), t = (int)(item % nt);
  const float r = e.rstd[row];
  float v[16], h[8];
  bsum16(e, row, t * 16, v);
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const float gt = v[c] * r, up = v[c + 8] * r;
    h[c] = gt / (1.0f + expf(-gt)) * up;
  }
  store_frag8(e.ahi, e.alo, row, t * 8, e.a_kt, h);
}

// QKV (block rows) and KVT (appended context rows): packed Q/K tiles hold 8 rotary pairs
// (m, m + hd/2) of one head; RoPE at the row's position; Q rows fp32, K and V to the
// row's sequence cache (fp16) at the row's slot.
__global__ void k_bqkv(BEpiArgs e, BRows rows) {
  const int nt_all = e.N / 16;
  const long item = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (item >= (long)e.M * nt_all) return;
  const int row = (int)(item / nt_all), t = (int)(item % nt_all);
  const int hd = e.hd, tph = hd / 16, half = hd / 2;
  const int q_tiles = e.q_tiles, kv_tiles = e.kv_tiles;
  int region, tt;  // 0 = Q, 1 = K, 2 = V
  if (t < q_tiles) {
    region = 0;
    tt = t;
  } else if (t < q_tiles + kv_tiles) {
    region = 1;
    tt = t - q_tiles;
  } else {
    region = 2;
    tt = t - q_tiles - kv_tiles;
  }
  const int head = tt / tph, jj = tt % tph;
  // the row's sequence, position and cache slot
  int i = 0;
  while (i + 1 < rows.n_seq && row >= rows.off[i + 1]) ++i;
  const int slot = rows.L[i] + (row - rows.off[i]);
  const long cache = (long)rows.seq[i] * e.seq_stride + (long)e.layer * e.cache_layer;
  const float r = e.rstd[row];
  float v[16];
  bsum16(e, row, t * 16, v);
#pragma unroll
  for (int c = 0; c < 16; ++c) v[c] *= r;
  if (region < 2) {
    const float2* cs = e.rope + (long)slot * half;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int m = 8 * jj + c;
      const float2 w = cs[m];
      const float a = v[c], b = v[c + 8];
      const float ya = a * w.x - b * w.y, yb = b * w.x + a * w.y;
      if (region == 0) {
        e.Q[(long)row * e.q_dim + head * hd + m] = ya;
        e.Q[(long)row * e.q_dim + head * hd + half + m] = yb;
      } else {
        uint16_t* k = e.kc + cache + ((long)head * e.Lcap + slot) * hd;
        k[m] = f2h(ya);
        k[half + m] = f2h(yb);
      }
    }
  } else {
#pragma unroll
    for (int c = 0; c < 16; ++c) {
      const int dim = jj * 16 + c;
      e.vt[cache + ((long)head * hd + dim) * e.Lcap + slot] = f2h(v[c]);
    }
  }
}

// ------------------------------------------------------------------------------------------
// attention over ragged contexts (Sec. 3.2: no mask; block rows see the whole context of
// their sequence and the whole block).  Item (sequence i of the call, chunk c, KV head g);
// 4 waves; wave w takes query tiles w, w + 4, ... of the G*B rows of head g, each against
// all keys of the chunk.  The chunk's K rows and V^T rows (fp16) are staged in LDS with
// XOR-swizzled 16-byte columns; scores are formed transposed (S^T = K Q^T) so that the
// probabilities are the B operand of the P V product.
// ------------------------------------------------------------------------------------------
template <int HD>
__global__ __launch_bounds__(256, 2) void k_battn(BAttnArgs a, BRows rows) {
  constexpr int CK = kChunk, CKM = CK + 32, NKB = CKM / 32;
  constexpr int KC = HD / 8, VC = CKM / 8;
  constexpr int KP = CKM * KC, VP = HD * VC;
  constexpr int NT = 256, PER = (KP + VP) / NT;
  static_assert((KP + VP) % NT == 0, "pieces split evenly");
  __shared__ u32x4 stage[KP + VP];
  u32x4* sK = stage;
  u32x4* sV = stage + KP;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  // item -> (sequence i, chunk c, head g)
  const int j = blockIdx.x;
  int i = 0;
  while (i + 1 < rows.n_seq && j >= rows.ipfx[i + 1]) ++i;
  const int L = rows.L[i];
  const int nch = max(1, (L + CK - 1) / CK);
  const int c = (j - rows.ipfx[i]) / a.n_kv, g = (j - rows.ipfx[i]) % a.n_kv;
  const int kbeg = c * CK;
  const int nkeys = ((c == nch - 1) ? L + a.B : kbeg + CK) - kbeg;
  const long cache = (long)rows.seq[i] * a.seq_stride + (long)a.layer * a.cache_layer;
  const uint16_t* kc = a.kc + cache;
  const uint16_t* vt = a.vt + cache;
  const int G = a.n_q / a.n_kv, R = G * a.B, QT = (R + 15) / 16;

  u32x4 pcs[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    pcs[k] = u32x4{0u, 0u, 0u, 0u};
    const int p = k * NT + tid;
    if (p < KP) {
      const int r = p / KC, col = p % KC;
      if (r < nkeys) pcs[k] = *reinterpret_cast<const u32x4*>(kc + ((long)g * a.Lcap + kbeg + r) * HD + col * 8);
    } else {
      const int pv = p - KP, d = pv / VC, col = pv % VC;
      if (col * 8 < nkeys)
        pcs[k] = *reinterpret_cast<const u32x4*>(vt + ((long)g * HD + d) * a.Lcap + kbeg + col * 8);
    }
  }
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int p = k * NT + tid;
    if (p < KP) {
      const int rr = p / KC, col = p % KC;
      sK[rr * KC + (col ^ (rr & 7))] = pcs[k];
    } else {
      const int pv = p - KP, d = pv / VC, col = pv % VC;
      u32x4 v = pcs[k];
      const int nv = nkeys - col * 8;  // values of keys past the end become zeros
      if (nv < 8) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (2 * e >= nv) v[e] = 0u;
          else if (2 * e + 1 >= nv) v[e] &= 0xFFFFu;
        }
      }
      sV[d * VC + (col ^ (d & 3))] = v;
    }
  }
  __syncthreads();

  const char* lds = reinterpret_cast<const char*>(stage);
  const int q = lane & 15, quad = lane >> 4;
  int k_at[HD / 32];
#pragma unroll
  for (int ks = 0; ks < HD / 32; ++ks) k_at[ks] = (q * KC + ((ks * 4 + quad) ^ (q & 7))) * 16;
  const int vx = (quad >> 1) ^ (q & 3);
  const int vbase = KP * 16 + (quad & 1) * 8;
  const int v0 = vbase + (q * VC + vx) * 16, v1 = vbase + (q * VC + (vx ^ 2)) * 16;
  const int q_dim = a.n_q * HD;
  const int nkb = (nkeys + 31) / 32;

  for (int qt = w; qt < QT; qt += 4) {
    const int r = qt * 16 + q;
    const bool rv = r < R;
    const int bb = rv ? r % a.B : 0;
    const int h = g * G + (rv ? r / a.B : 0);
    const float* src = a.Q + (long)(rows.off[i] + bb) * q_dim + h * HD;
    u32x4 qh[HD / 32], ql[HD / 32];
#pragma unroll
    for (int ks = 0; ks < HD / 32; ++ks) {
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = rv ? src[ks * 32 + quad * 8 + e] * a.qscale : 0.f;
      split_pack8_h(v, qh[ks], ql[ks]);
    }
    f32x4 sc[2 * NKB];
#pragma unroll
    for (int kk = 0; kk < NKB; ++kk) {
      f32x4 a0 = {-INFINITY, -INFINITY, -INFINITY, -INFINITY}, a1 = a0;
      if (kk < nkb) {
        f32x4 h0 = {0.f, 0.f, 0.f, 0.f}, l0 = h0, h1 = h0, l1 = h0;
#pragma unroll
        for (int ks = 0; ks < HD / 32; ++ks) {
          const u32x4 k0v = *reinterpret_cast<const u32x4*>(lds + k_at[ks] + (2 * kk) * 16 * KC * 16);
          const u32x4 k1v = *reinterpret_cast<const u32x4*>(lds + k_at[ks] + (2 * kk + 1) * 16 * KC * 16);
          h0 = mfma_h(k0v, qh[ks], h0);
          h1 = mfma_h(k1v, qh[ks], h1);
          l0 = mfma_h(k0v, ql[ks], l0);
          l1 = mfma_h(k1v, ql[ks], l1);
        }
        a0 = h0 + l0;
        a1 = h1 + l1;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (2 * kk * 16 + quad * 4 + e >= nkeys) a0[e] = -INFINITY;
          if ((2 * kk + 1) * 16 + quad * 4 + e >= nkeys) a1[e] = -INFINITY;
        }
      }
      sc[2 * kk] = a0;
      sc[2 * kk + 1] = a1;
    }
    float m = -INFINITY, l = 0.f;
#pragma unroll
    for (int kt = 0; kt < 2 * NKB; ++kt)
#pragma unroll
      for (int e = 0; e < 4; ++e) m = fmaxf(m, sc[kt][e]);
    m = fmaxf(m, __shfl_xor(m, 16));
    m = fmaxf(m, __shfl_xor(m, 32));
#pragma unroll
    for (int kt = 0; kt < 2 * NKB; ++kt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p = exp2f(sc[kt][e] - m);
        sc[kt][e] = p;
        l += p;
      }
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    f32x4 o[HD / 16];
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < NKB; ++kk) {
      if (kk < nkb) {
        float pv[8] = {sc[2 * kk][0], sc[2 * kk][1], sc[2 * kk][2], sc[2 * kk][3],
                       sc[2 * kk + 1][0], sc[2 * kk + 1][1], sc[2 * kk + 1][2], sc[2 * kk + 1][3]};
        u32x4 ph, pl;
        split_pack8_h(pv, ph, pl);
#pragma unroll
        for (int dt = 0; dt < HD / 16; ++dt) {
          const int off = (dt * 16 * VC + kk * 4) * 16;
          const u32x2 x0 = *reinterpret_cast<const u32x2*>(lds + v0 + off);
          const u32x2 x1 = *reinterpret_cast<const u32x2*>(lds + v1 + off);
          const u32x4 vv = {x0[0], x0[1], x1[0], x1[1]};
          o[dt] = mfma_h(vv, ph, o[dt]);
          o[dt] = mfma_h(vv, pl, o[dt]);
        }
      }
    }
    if (rv) {
      const long base = (long)j * a.Rpad + r;
#pragma unroll
      for (int dt = 0; dt < HD / 16; ++dt)
        *reinterpret_cast<f32x4*>(a.OP + base * HD + dt * 16 + quad * 4) = o[dt];
      if (quad == 0) a.ML[base] = make_float2(m, l);
    }
  }
}

// merge the chunk partials of query row r of head g of sequence i (one wave per row) and
// write the A fragments of the output projection at row off[i] + r % B
template <int HD>
__global__ __launch_bounds__(64) void k_bcomb(BAttnArgs a, BRows rows, u32x4* ohi, u32x4* olo, int a_kt) {
  constexpr int DPL = HD / 64;
  const int lane = threadIdx.x;
  const int G = a.n_q / a.n_kv, R = G * a.B;
  const int it = blockIdx.x;
  const int i = it / (a.n_kv * R), g = (it / R) % a.n_kv, r = it % R;
  if (i >= rows.n_seq) return;
  const int nch = max(1, (rows.L[i] + kChunk - 1) / kChunk);
  const long jb = rows.ipfx[i] + g;  // item of chunk 0; chunk c at jb + c * n_kv
  float M = -INFINITY;
  for (int c = lane; c < nch; c += 64) M = fmaxf(M, a.ML[(jb + (long)c * a.n_kv) * a.Rpad + r].x);
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) M = fmaxf(M, __shfl_xor(M, off));
  float num[DPL], den = 0.f;
#pragma unroll
  for (int e = 0; e < DPL; ++e) num[e] = 0.f;
  for (int c = 0; c < nch; ++c) {
    const long base = (jb + (long)c * a.n_kv) * a.Rpad + r;
    const float2 mc = a.ML[base];
    const float wgt = exp2f(mc.x - M);
    den += wgt * mc.y;
#pragma unroll
    for (int e = 0; e < DPL; ++e) num[e] += wgt * a.OP[base * HD + lane * DPL + e];
  }
  const float inv = 1.0f / den;
  const int row = rows.off[i] + r % a.B, h = g * G + r / a.B;
  uint32_t* hi = reinterpret_cast<uint32_t*>(ohi);
  uint32_t* lo = reinterpret_cast<uint32_t*>(olo);
  if constexpr (DPL == 2) {
    store_frag_pair(hi, lo, row, h * HD + 2 * lane, a_kt, num[0] * inv, num[1] * inv);
  } else {
    const float y = num[0] * inv, y1 = __shfl_xor(y, 1);
    if ((lane & 1) == 0) store_frag_pair(hi, lo, row, h * HD + lane, a_kt, y, y1);
  }
}

// ------------------------------------------------------------------------------------------
// launchers
// ------------------------------------------------------------------------------------------
int bgemm_groups(int Nt, int Mt) { return ((Nt + kBN - 1) / kBN) * ((Mt + kBM - 1) / kBM); }

void launch_bgemm(hipStream_t s, const BGemmArgs& g, bool argmax) {
  const dim3 grid(bgemm_groups(g.Nt, g.Mt) * g.kg);
  if (argmax) hipLaunchKernelGGL(k_bgemm<true>, grid, dim3(kBT), 0, s, g);
  else hipLaunchKernelGGL(k_bgemm<false>, grid, dim3(kBT), 0, s, g);
}

void launch_bargmax(hipStream_t s, const float* pmax, const int* pidx, int ngroups, int pld, int M, int* tokens) {
  hipLaunchKernelGGL(k_bargmax, dim3(M), dim3(64), 0, s, pmax, pidx, ngroups, pld, M, tokens);
}

void launch_brstd(hipStream_t s, const float* stats, int n_st, int M, float inv_dim, float eps, float* rstd) {
  hipLaunchKernelGGL(k_brstd, dim3(M), dim3(64), 0, s, stats, n_st, M, inv_dim, eps, rstd);
}

static int blocks_for(long items) { return (int)((items + 255) / 256); }

void launch_bembed(hipStream_t s, const uint16_t* embed, const int32_t* ids, int M, int H, int V,
                   const float* gain, float* X, float* stats, u32x4* ahi, u32x4* alo, int a_kt) {
  hipLaunchKernelGGL(k_bembed, dim3(blocks_for((long)M * (H / 16))), dim3(256), 0, s, embed, ids, M, H, V, gain, X,
                     stats, ahi, alo, a_kt);
}

void launch_bepi(hipStream_t s, int kind, const BEpiArgs& e, const BRows& rows) {
  switch (kind) {
    case BEPI_RESID:
      hipLaunchKernelGGL(k_bresid, dim3(blocks_for((long)e.M * (e.H / 16))), dim3(256), 0, s, e);
      break;
    case BEPI_SWIGLU:
      hipLaunchKernelGGL(k_bswiglu, dim3(blocks_for((long)e.M * (e.N / 16))), dim3(256), 0, s, e);
      break;
    default:
      hipLaunchKernelGGL(k_bqkv, dim3(blocks_for((long)e.M * (e.N / 16))), dim3(256), 0, s, e, rows);
      break;
  }
}

void launch_battn(hipStream_t s, int hd, const BAttnArgs& a, const BRows& rows, int items) {
  if (hd == 64) hipLaunchKernelGGL(k_battn<64>, dim3(items), dim3(256), 0, s, a, rows);
  else hipLaunchKernelGGL(k_battn<128>, dim3(items), dim3(256), 0, s, a, rows);
}

void launch_bcomb(hipStream_t s, int hd, const BAttnArgs& a, const BRows& rows, u32x4* ohi, u32x4* olo, int a_kt) {
  const int R = (a.n_q / a.n_kv) * a.B;
  const dim3 grid(rows.n_seq * a.n_kv * R);
  if (hd == 64) hipLaunchKernelGGL(k_bcomb<64>, grid, dim3(64), 0, s, a, rows, ohi, olo, a_kt);
  else hipLaunchKernelGGL(k_bcomb<128>, grid, dim3(64), 0, s, a, rows, ohi, olo, a_kt);
}

}  // namespace dflare
