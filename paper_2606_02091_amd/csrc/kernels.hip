// HIP kernels of the DFlare draft step for gfx950 (CDNA4, wave64, MFMA).
//
// Data types: weights, embeddings and the KV cache are bf16; activations, the
// residual stream and every accumulation are fp32.  Activations enter the bf16
// matrix cores as an exact-sum pair hi + lo of bf16 values (hi = bf16(x),
// lo = bf16(x - hi)), so each product carries about 16 mantissa bits of the
// activation against the exact bf16 weight; the doubled MFMA work is free
// because every GEMM here streams its weights from HBM (batch-1, 16 rows).
//
// A draft block (Sec. 3.2, Eq. 4, and the LM head) runs as one persistent launch of one
// 8-wave work-group per CU.  Its phases are separated by grid barriers, and each phase
// issues the loads that do not depend on the previous phase (its first weight tiles, the
// context K/V of attention) before it waits, so HBM keeps streaming across the barrier.
//
// Cross-phase data and the per-XCD L2 caches.  Each XCD has its own L2, and ordinary
// stores stay in the writer's L2 until the kernel ends.  So within a launch:
//   - everything a later phase reads is stored write-through (agent-scope atomic stores,
//     which reach the device-coherent level before they complete), and every work-group
//     waits for its stores before it arrives at a barrier;
//   - a line is read with ordinary (L2-cached) loads only if it is written at most once
//     per launch, before any read of it: the per-stage and per-layer buffers below.  At
//     launch start the L2s hold no copy of such a line, so the first read fetches the
//     written value.  Buffers that are rewritten within a launch (the residual stream,
//     the attention partials, the LM-head maxima) are read with coherent loads.
#include <math.h>

#include "device_common.h"

namespace dflare {

constexpr long long kBarrierTimeout = 25000000;  // wall-clock ticks (100 MHz): 0.25 s

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
// layer fusion (Eq. 3): u^(i)[r, k] = sum_j alpha[i, j] h^(j)[r, k], accumulated in j order.
// Block (512 columns, row r, draft layer i); a lane owns 8 columns and keeps up to forty
// 16-byte loads in flight (every target layer at once for S <= 40: one memory round trip).
// Writes the A fragments of u^(i) * g_fuse^(i) and per-16-column sums of squares of u^(i);
// the 1/rms of Eq. 3 is applied in the K/V projection.  The D blocks of one (512 columns,
// row) pair read the same target row pieces; consecutive block ids are dealt to the 8 XCDs
// in turn, so the pair's D blocks get ids 8 apart (one XCD, one L2), where they can share
// the pieces.  Ids past the last pair are idle.
// ------------------------------------------------------------------------------------------
constexpr int kFuseBatch = 40;  // target layers whose loads are in flight together
constexpr int kXcds = 8;
__global__ __launch_bounds__(64) void k_fuse(const uint16_t* __restrict__ hidden, int ld, int S, int H, int n, int D,
                                             const float* __restrict__ alpha, const float* __restrict__ gain,
                                             float* ustats, u32x4* ua_hi, u32x4* ua_lo, int n_max, int mt_max) {
  const int lane = threadIdx.x;
  // block id b = x + 8 (i + D g): pair m = 8 g + x (x = b % 8), draft layer i
  const int b = blockIdx.x, x = b % kXcds, i = (b / kXcds) % D, m = kXcds * (b / (kXcds * D)) + x;
  const int cbs = (H + 511) / 512;
  if (m >= cbs * n) return;
  const int r = m / cbs, cb = m % cbs;
  const int k0 = cb * 512 + lane * 8;
  const bool ok = k0 < H;
  const int Kt = H / 32;
  float u[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int j0 = 0; j0 < S; j0 += kFuseBatch) {
    u32x4 v[kFuseBatch];
#pragma unroll
    for (int qq = 0; qq < kFuseBatch; ++qq) {
      v[qq] = u32x4{0u, 0u, 0u, 0u};
      if (ok && j0 + qq < S) v[qq] = *reinterpret_cast<const u32x4*>(hidden + ((long)(j0 + qq) * ld + r) * H + k0);
    }
#pragma unroll
    for (int qq = 0; qq < kFuseBatch; ++qq) {
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
// context K/V projection of fuse_append (Eq. 4, W^t): RoPE(f W_K^t) and f W_V^t for every
// appended row of every draft layer, into cache slots L + row.  Weight-streaming GEMM:
// block (group of NT output tiles, layer, 16-row m-tile); its WAVES waves split the k range
// and add their partial sums in LDS in wave order.  Two register sets alternate so that one
// batch of loads is in flight while the previous one goes through the matrix cores.
// ------------------------------------------------------------------------------------------
template <int NT, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void k_kvt(KvtArgs a) {
  constexpr int U = 2;  // k-tiles per batch
  __shared__ f32x4 red[WAVES][NT][64];
  __shared__ float s_rstd[16];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int quad = lane >> 4, col = lane & 15;
  const int group = blockIdx.x;
  const int layer = blockIdx.y, mt = blockIdx.z;
  const int M = a.n_new;
  if (mt * 16 >= M) return;  // whole m-tile idle: every block of it leaves together

  const int kw0 = (a.Kt * wave) / WAVES;
  const int nk = (a.Kt * (wave + 1)) / WAVES - kw0;
  const int nb = (nk + U - 1) / U;
  const int nb2 = (nb + 1) & ~1;
  const int nt0 = group * NT;

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

#pragma unroll
  for (int j = 0; j < NT; ++j) red[wave][j][lane] = acc_h[j] + acc_l[j];
  __syncthreads();
  const bool owner = wave < NT;
  const int nt = nt0 + (owner ? wave : 0);
  const bool has_tile = owner && nt < a.Nt;
  f32x4 v = {0.f, 0.f, 0.f, 0.f};
  if (owner) {
    v = red[0][wave][lane];
#pragma unroll
    for (int w = 1; w < WAVES; ++w) v += red[w][wave][lane];
  }
  // 1/rms of the fused rows (Eq. 3): (u*g/rms) W^T = (1/rms) (u*g) W^T
  if (tid < 256) {
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
    if (part == 0) s_rstd[row] = (mt * 16 + row < M) ? rsqrtf(s * a.inv_dim + a.eps) : 0.f;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] *= s_rstd[quad * 4 + i];

  if (has_tile) {
    const int tph = a.hd / 16, half = a.hd / 2;
    const int L0 = a.Lp ? *a.Lp : a.L;  // rows go to cache slots L0 + row
    uint16_t* kc = a.kc + layer * a.cache_layer_stride;
    uint16_t* vt = a.vt + layer * a.cache_layer_stride;
    const bool is_k = nt < a.kv_tiles;
    const int t = is_k ? nt : nt - a.kv_tiles;
    const int head = t / tph, jj = t % tph;
    // bias of this lane's column (K columns are packed in rotary pair order)
    const int kvd = a.kv_tiles * 16;
    const int kdim = (col < 8) ? 8 * jj + (col & 7) : half + 8 * jj + (col & 7);
    const float bcol =
        a.bias ? a.bias[(long)layer * 2 * kvd + (is_k ? head * a.hd + kdim : kvd + head * a.hd + jj * 16 + col)] : 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = mt * 16 + quad * 4 + i;
      const bool valid = row < M;
      const int slot = L0 + row;
      const float x = v[i] + bcol;
      const float partner = __shfl_xor(x, 8);
      if (is_k) {
        const int m = 8 * jj + (col & 7);
        const int dim = (col < 8) ? m : half + m;
        const float2 cs = a.rope[(long)(valid ? slot : 0) * half + m];
        const float y = (col < 8) ? (x * cs.x - partner * cs.y) : (x * cs.x + partner * cs.y);
        if (valid) kc[((long)head * a.Lcap + slot) * a.hd + dim] = f2h(y);
      } else if (valid) {
        const int dim = jj * 16 + col;
        vt[((long)head * a.hd + dim) * a.Lcap + slot] = f2h(x);
      }
    }
  }
}

// ---- init: folding a linear layer into the next one (the +FC variant) ----
// out = A B for bf16 row-major A [R, O] and B [O, K], in double precision.  Work-group:
// a 64 x 64 tile of out, 256 threads with 4 x 4 outputs each; 16-deep slices of A and B
// staged in LDS as doubles.
__global__ __launch_bounds__(256) void k_compose(uint16_t* out, const uint16_t* A, const uint16_t* B, int R, int O,
                                                 int K) {
  __shared__ double sa[16][65];
  __shared__ double sb[16][65];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  double acc[4][4] = {};
  for (int o0 = 0; o0 < O; o0 += 16) {
    for (int i = threadIdx.x; i < 16 * 64; i += 256) {
      const int oo = i & 15, rr = i >> 4;  // A: row r0 + rr, column o0 + oo
      sa[oo][rr] = (r0 + rr < R && o0 + oo < O) ? (double)bf2f(A[(long)(r0 + rr) * O + o0 + oo]) : 0.0;
      const int cc = i & 63, ob = i >> 6;  // B: row o0 + ob, column c0 + cc
      sb[ob][cc] = (o0 + ob < O && c0 + cc < K) ? (double)bf2f(B[(long)(o0 + ob) * K + c0 + cc]) : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int oo = 0; oo < 16; ++oo)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += sa[oo][ty * 4 + i] * sb[oo][tx * 4 + j];
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = r0 + ty * 4 + i, c = c0 + tx * 4 + j;
      if (r < R && c < K) out[(long)r * K + c] = f2bf((float)acc[i][j]);
    }
}

// y = A b in double precision: one work-group of 256 per output row
__global__ __launch_bounds__(256) void k_matvec(float* y, const uint16_t* A, const uint16_t* b, int O) {
  __shared__ double red[256];
  const int r = blockIdx.x;
  double s = 0.0;
  if (b)
    for (int o = threadIdx.x; o < O; o += 256) s += (double)bf2f(A[(long)r * O + o]) * (double)bf2f(b[o]);
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) y[r] = (float)red[0];
}

// ==========================================================================================
// the draft block
// ==========================================================================================

// The draft kernel reads its fixed arguments through the constant address space: they are
// never written during a launch, so every field is a scalar load where a phase uses it.
typedef const CONSTANT DraftArgs* Args;
typedef const CONSTANT DraftCall* Call;

// The work-group's barrier-failure flag lives in LDS (written and read by wave 0 only): a
// flag in private memory would be read with a vector load, which completes only after every
// load the wave issued before it, so a poll behind weight requests could not start early.
typedef volatile LDSP int* Failed;
constexpr int kFailOff = 80 * 1024 - 16;  // just below the attention staging area

// ---- grid barrier ----
// Arrival: every wave waits for its own stores, then one atomic add per work-group on one
// of kBarCounters counters (spreading the arrivals keeps same-address atomics from
// serialising).  Wait: lanes of wave 0 poll the counters with coherent loads until each
// holds its share of arrivals times the barrier's epoch.  A wait that exceeds the time
// limit raises the host-visible error flag and lets the work-group go on (results are then
// wrong, and the host reports the failure), so a launch always terminates.
__device__ __forceinline__ void grid_arrive(Args a, bool wait_own = true) {
  if (wait_own) wait_vm();
  __syncthreads();
  if (threadIdx.x == 0)
    __hip_atomic_fetch_add(a->bar + (blockIdx.x % kBarCounters) * 32, 1u, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void trace_mark(Call c, int slot, int nslots) {
  if (c->trace && threadIdx.x == 0) c->trace[(long)blockIdx.x * nslots + slot] = wall_clock64();
}

__device__ __forceinline__ void grid_wait(Args a, unsigned epoch, Failed failed) {
  if (threadIdx.x < 64 && !*failed) {
    const int lane = threadIdx.x;
    const unsigned n = gridDim.x;
    const unsigned share = n / kBarCounters + ((unsigned)lane < n % kBarCounters ? 1u : 0u);
    const unsigned target = share * epoch;
    unsigned* c = a->bar + (lane % kBarCounters) * 32;
    const long long t0 = wall_clock64();
    while (true) {
      const bool ok = lane >= kBarCounters ||
                      __hip_atomic_load(c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= target;
      if (__all(ok)) break;
      __builtin_amdgcn_s_sleep(1);
      if (wall_clock64() - t0 > kBarrierTimeout) {
        if (lane == 0) {
          *failed = 1;
          __hip_atomic_store(a->err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        }
        break;
      }
    }
  }
  __syncthreads();
}

struct PhaseCtl {
  bool wait;        // wait at the grid barrier before the phase body
  unsigned epoch;   // that barrier's epoch
  int slot, nslots; // trace slot of the body start
};

__device__ __forceinline__ void phase_begin(Args a, Call c, const PhaseCtl& pc,
                                            Failed failed) {
  if (pc.wait) grid_wait(a, pc.epoch, failed);
  trace_mark(c, pc.slot, pc.nslots);
}

// Q/K/V -> attention hand-over without a grid barrier.  An attention item of KV head g needs
// only the Q tiles of g's query heads and g's K and V tiles (its block keys), (G + 2) hd / 16
// tiles per layer.  Each work-group that finishes Q/K/V tiles (a range's first work-group, or
// every one without a K split) adds, once every wave's stores are complete, the number it
// finished of each head to that head's counter; an item waits until its head's counter holds
// this layer's count (counters are monotonic across launches, from qcnt_base).
__device__ __forceinline__ void qkv_arrive(Args a) {
  wait_vm();
  __syncthreads();
  if (threadIdx.x == 0) {
    const int kg = a->kg[PH_QKV];
    if (blockIdx.x % kg == 0) {
      const int rg = blockIdx.x / kg, nq = a->nq[PH_QKV], nr = a->nr[PH_QKV];
      const int t0 = rg * nq + min(rg, nr), t1 = t0 + nq + (rg < nr ? 1 : 0);
      const int tph = a->hd / 16, G = a->n_q / a->n_kv, nqt = a->n_q * tph, nkt = a->n_kv * tph;
      int head = -1;
      unsigned n = 0;
      for (int t = t0; t < t1; ++t) {
        const int hq = t < nqt ? t / (G * tph) : (t - nqt < nkt ? (t - nqt) / tph : (t - nqt - nkt) / tph);
        if (hq != head) {
          if (n) __hip_atomic_fetch_add(a->qcnt + head * 32, n, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          head = hq;
          n = 0;
        }
        ++n;
      }
      if (n) __hip_atomic_fetch_add(a->qcnt + head * 32, n, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

__device__ __forceinline__ void qkv_wait(Args a, Call c, int layer, int g, Failed failed) {
  if (threadIdx.x < 64 && !*failed) {
    const unsigned* cnt = a->qcnt + g * 32;
    const unsigned target =
        c->qcnt_base + (unsigned)(layer + 1) * (unsigned)((a->n_q / a->n_kv + 2) * (a->hd / 16));
    const long long t0 = wall_clock64();
    while (__hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      __builtin_amdgcn_s_sleep(1);
      if (wall_clock64() - t0 > kBarrierTimeout) {
        if (threadIdx.x == 0) {
          *failed = 1;
          __hip_atomic_store(a->err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        }
        break;
      }
    }
  }
  __syncthreads();
}

// Context length of the call: the host's value or, when the length is kept on the device
// (after a verification step that did not wait), the word written by that step.
__device__ __forceinline__ int ctx_len(Call c) { return c->Lp ? *c->Lp : c->L; }

// ---- EMBED: X = E[ids] (fp32), sums of squares and A fragments of X * g_attn^(0) (stage 0)
// Run by wave 0.  Item = 8 columns of one row; items 2m and 2m + 1 (one 16-column tile) go to
// lanes 2k and 2k + 1 of work-group m % blocks, so the work spreads over every work-group and
// the two halves of a tile meet in one shuffle.
__device__ __forceinline__ void phase_embed(Args a, Call c) {
  const int H = a->H, Kt = H / 32, per_row = H / 8;
  const int pairs = a->B * per_row / 2;
  const float* gain = a->g_attn;
  float* XS = a->XS;
  uint32_t* xhi = reinterpret_cast<uint32_t*>(a->XA);
  uint32_t* xlo = reinterpret_cast<uint32_t*>(a->XA + (long)(Kt + kKtPad) * 64);
  const int tid = opaque(threadIdx.x);  // threads of wave 0
  for (int m = blockIdx.x + (tid >> 1) * gridDim.x; m < pairs; m += 32 * gridDim.x) {
    const int item = 2 * m + (tid & 1);
    const int row = item / per_row, k0 = (item % per_row) * 8;
    int id = gbl(c->ids)[row];
    id = id < 0 ? 0 : (id >= a->V ? a->V - 1 : id);
    const u32x4 v = *gbl(reinterpret_cast<const u32x4*>(a->embed + (long)id * H + k0));
    float f[8], y[8], sq = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[2 * e] = bf2f(v[e] & 0xFFFFu);
      f[2 * e + 1] = bf2f(v[e] >> 16);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      sq += f[e] * f[e];
      y[e] = f[e] * gbl(gain)[k0 + e];
    }
    sq += __shfl_xor(sq, 1);
    float* xo = a->X + (long)row * H + k0;
    st_wt16(xo, u32x4{__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]), __float_as_uint(f[3])});
    st_wt16(xo + 4, u32x4{__float_as_uint(f[4]), __float_as_uint(f[5]), __float_as_uint(f[6]), __float_as_uint(f[7])});
    u32x4 hi, lo;
    split_pack8(y, hi, lo);
    const long fo = frag_off(row, k0, Kt);  // in bf16 elements
    st_wt16(reinterpret_cast<uint16_t*>(xhi) + fo, hi);
    st_wt16(reinterpret_cast<uint16_t*>(xlo) + fo, lo);
    if ((item & 1) == 0) st_wt(XS + (k0 / 16) * kStatsPad + row, sq);
  }
}

// ---- weight-streaming GEMM phases ----
enum Epi { EPI_RESID = 0, EPI_SWIGLU = 1, EPI_QKV = 2, EPI_ARGMAX = 3 };

struct GemmJob {
  const u32x4* W;      // packed tiles of this layer
  int Nt, Kt;
  const u32x4* Ahi;    // A fragments of the input rows (one 16-row tile)
  const u32x4* Alo;
  const float* stats;  // sums of squares [H/16][kStatsPad] of an RMSNorm input, or null
  // RESID
  float* xs_out;       // [H/16][kStatsPad]
  uint32_t* na_hi;     // A fragments of the next consumer
  uint32_t* na_lo;
  int na_Kt;
  const float* gain;   // RESID: gain of the next RMSNorm
  float* hid_out;      // RESID after the MLP: optional copy of the layer's output rows [B, H]
  // QKV
  float* q_out;        // [16, q_dim]
  uint16_t* kc;        // cache of this layer
  uint16_t* vt;
  // split-K
  float* part;         // partial tiles of this phase kind [blocks][kTNMax][64 lanes][4]
  unsigned tag;        // low mantissa bit every partial of this use carries
};

// LDS of a GEMM phase: partial tiles [kWaves][TN][64 lanes] (64 KiB at most), then the
// row scales, the argmax scratch and a flag.
constexpr int kLdsRedBytes = kWaves * kTNMax * 1024;
// LDS of the attention phase: the merge area at 0 (shared with the GEMM reduction area), the
// K / V^T staging area from kStageOff to the end.  GEMM phases never touch the staging
// area, so the next layer's context pieces can be streamed into it during them.
constexpr int kStageOff = 80 * 1024;
static_assert(kLdsRedBytes + 2048 <= kFailOff && kFailOff + 16 == kStageOff,
              "GEMM scratch, the failure flag and the attention staging area do not overlap");


// Inputs of a tile's epilogue that do not depend on its sums: the residual rows and the next
// norm's gain (RESID), the rotary (cos, sin) of the lane's rows (Q and K tiles of QKV).  They
// are loaded before the tile's sums are complete, so that their latency overlaps the waves'
// reduction and the wait for the split-K partials.  (The residual rows were last written in
// an earlier phase, before a grid barrier.)
struct EpiIn {
  float x[4];
  float gn;
  float2 cs[4];
};
template <int EPI>
__device__ __forceinline__ EpiIn epilogue_inputs(Args a, Call c, const GemmJob& g, int nt) {
  EpiIn in{};
  const int lane = opaque(threadIdx.x) & 63;
  const int quad = lane >> 4, col = lane & 15;
  const int M = a->B;
  if constexpr (EPI == EPI_RESID) {
    const int k = nt * 16 + col;
    in.gn = gbl(g.gain)[k];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = quad * 4 + i;
      in.x[i] = row < M ? ld_coh(a->X + (long)row * a->H + k) : 0.f;
    }
  } else if constexpr (EPI == EPI_QKV) {
    const int hd = a->hd, tph = hd / 16, half = hd / 2;
    if (nt < (a->n_q + a->n_kv) * tph) {  // Q and K tiles (tph divides the Q tile count)
      const int L = ctx_len(c);
      const int m = 8 * (nt % tph) + (col & 7);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = quad * 4 + i;
        const int pos = row < M ? c->pos[row] + (c->Lp ? L : 0) : 0;
        const uint64_t csb = gbl(reinterpret_cast<const uint64_t*>(a->rope))[(long)pos * half + m];
        in.cs[i] = make_float2(__uint_as_float((uint32_t)csb), __uint_as_float((uint32_t)(csb >> 32)));
      }
    }
  }
  return in;
}

// Epilogue of one finished 16 x 16 output tile nt (lane holds rows quad*4 .. +3 of column
// col); v already carries the RMSNorm row scale, `in` the tile's epilogue_inputs.  ARGMAX
// leaves the tile's best (logit, id) per row in s_bv / s_bi at slot j.
template <int EPI>
__device__ __forceinline__ void gemm_epilogue(Args a, Call c, const GemmJob& g, int nt, f32x4 v, const EpiIn& in,
                                              int j, float* s_bv, int* s_bi) {
  const int lane = opaque(threadIdx.x) & 63;  // epilogue values are not hoisted above the main loop
  const int quad = lane >> 4, col = lane & 15;
  const int M = a->B;
  if constexpr (EPI == EPI_RESID) {
    const int k = nt * 16 + col;
    const float gn = in.gn;
    float sq[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = quad * 4 + i;
      float x = 0.f;
      if (row < M) {
        float* p = a->X + (long)row * a->H + k;
        x = in.x[i] + v[i];
        st_wt(p, x);
        if (g.hid_out) st_wt(g.hid_out + (long)row * a->H + k, x);
      }
      sq[i] = x * x;
      const float y = x * gn;
      const float y1 = __shfl_xor(y, 1);
      if ((col & 1) == 0 && row < M) store_frag_pair_wt(g.na_hi, g.na_lo, row, k, g.na_Kt, y, y1);
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
      for (int i = 0; i < 4; ++i) st_wt(g.xs_out + nt * kStatsPad + quad * 4 + i, sq[i]);
  } else if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float gt = v[i];
      const float up = __shfl_xor(gt, 8);
      const float hv = (col < 8) ? gt / (1.0f + expf(-gt)) * up : 0.f;
      const float h1 = __shfl_xor(hv, 1);
      const int row = quad * 4 + i;
      if (col < 8 && (col & 1) == 0 && row < M) store_frag_pair_wt(g.na_hi, g.na_lo, row, nt * 8 + col, g.na_Kt, hv, h1);
    }
  } else if constexpr (EPI == EPI_QKV) {
    const int L = ctx_len(c), hd = a->hd;
    const int tph = hd / 16, half = hd / 2;
    const int q_tiles = a->n_q * tph, kv_tiles = a->n_kv * tph;
    int region, t;  // 0 = Q, 1 = K, 2 = V
    if (nt < q_tiles) {
      region = 0;
      t = nt;
    } else if (nt < q_tiles + kv_tiles) {
      region = 1;
      t = nt - q_tiles;
    } else {
      region = 2;
      t = nt - q_tiles - kv_tiles;
    }
    const int head = t / tph, jj = t % tph;
    const int q_dim = a->n_q * hd;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = quad * 4 + i;
      const bool valid = row < M;
      const int slot = L + row;
      const float x = v[i];
      const float partner = __shfl_xor(x, 8);
      if (region < 2) {
        const int m = 8 * jj + (col & 7);
        const int dim = (col < 8) ? m : half + m;
        const float2 cs = in.cs[i];
        const float y = (col < 8) ? (x * cs.x - partner * cs.y) : (x * cs.x + partner * cs.y);
        if (valid) {
          if (region == 0) {
            st_wt(g.q_out + (long)row * q_dim + head * hd + dim, y);
          } else {  // block keys go to cache slots L + row
            st_wt(g.kc + ((long)head * a->Lcap + slot) * hd + dim, f2h(y));
          }
        }
      } else if (valid) {
        const int dim = jj * 16 + col;
        st_wt(g.vt + ((long)head * hd + dim) * a->Lcap + slot, f2h(x));
      }
    }
  } else if constexpr (EPI == EPI_ARGMAX) {
    const int vc = nt * 16 + col;
    const bool ok = vc < a->V;
    float bv[4];
    int bix[4];
    // sampling: the Gumbel-max score z / T + noise; the lane's rows 4 quad .. 4 quad + 3 are
    // block positions of one Philox call (sequence slot 0).  The logits stay unperturbed.
    const float inv_temp = c->inv_temp;
    float noise[4] = {0.f, 0.f, 0.f, 0.f};
    if (inv_temp > 0.f) gumbel_noise4(c->seed, vc, quad, c->draw, 0, noise);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = quad * 4 + i;
      if (ok && c->logits && row < M) c->logits[(long)row * a->V + vc] = v[i];
      const float y = (inv_temp > 0.f) ? v[i] * inv_temp + noise[i] : v[i];
      bv[i] = ok ? y : -INFINITY;
      bix[i] = ok ? vc : 0x7FFFFFFF;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) {
        const float ov = __shfl_xor(bv[i], off);
        const int oi = __shfl_xor(bix[i], off);
        if (ov > bv[i] || (ov == bv[i] && oi < bix[i])) {
          bv[i] = ov;
          bix[i] = oi;
        }
      }
    if (col == 0)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        s_bv[j * 16 + quad * 4 + i] = bv[i];
        s_bi[j * 16 + quad * 4 + i] = bix[i];
      }
  }
}

__host__ __device__ constexpr int gemm_ns(int TN) { return TN >= 8 ? 2 : 4; }  // steps in flight

// The GEMM job of phase (kind, layer): weights, input fragments and epilogue targets.
__device__ __forceinline__ GemmJob make_job(Args a, Call c, int kind, int layer) {
  GemmJob g{};
  const int H = a->H, Kt_H = H / 32, q_Kt = a->n_q * a->hd / 32, F_Kt = a->F / 32;
  switch (kind) {
    case PH_QKV: {
      const int s = 2 * layer;
      g.W = a->w_qkv + layer * a->s_qkv;
      g.Nt = (a->n_q + 2 * a->n_kv) * a->hd / 16;
      g.Kt = Kt_H;
      g.Ahi = a->XA + s * a->xa_stride;
      g.Alo = g.Ahi + (long)(Kt_H + kKtPad) * 64;
      g.stats = a->XS + s * a->xs_stride;
      g.q_out = a->Q + layer * a->q_stride;
      g.kc = a->kc + layer * a->cache_layer;
      g.vt = a->vt + layer * a->cache_layer;
      break;
    }
    case PH_O:
    case PH_DOWN: {
      const bool o = kind == PH_O;
      const int s = o ? 2 * layer + 1 : 2 * layer + 2;
      g.W = o ? a->w_o + layer * a->s_o : a->w_down + layer * a->s_down;
      g.Nt = H / 16;
      g.Kt = o ? q_Kt : F_Kt;
      g.Ahi = o ? a->OA + layer * a->oa_stride : a->HA + layer * a->ha_stride;
      g.Alo = g.Ahi + (long)(g.Kt + kKtPad) * 64;
      g.stats = nullptr;
      g.xs_out = a->XS + s * a->xs_stride;
      g.na_hi = reinterpret_cast<uint32_t*>(a->XA + s * a->xa_stride);
      g.na_lo = reinterpret_cast<uint32_t*>(a->XA + s * a->xa_stride + (long)(Kt_H + kKtPad) * 64);
      g.na_Kt = Kt_H;
      g.gain = o ? a->g_mlp + (long)layer * H : (layer + 1 < a->D ? a->g_attn + (long)(layer + 1) * H : a->g_final);
      g.hid_out = (!o && c->hidden) ? c->hidden + (long)layer * a->B * H : nullptr;
      break;
    }
    case PH_GU: {
      const int s = 2 * layer + 1;
      g.W = a->w_gu + layer * a->s_gu;
      g.Nt = 2 * a->F / 16;
      g.Kt = Kt_H;
      g.Ahi = a->XA + s * a->xa_stride;
      g.Alo = g.Ahi + (long)(Kt_H + kKtPad) * 64;
      g.stats = a->XS + s * a->xs_stride;
      g.na_hi = reinterpret_cast<uint32_t*>(a->HA + layer * a->ha_stride);
      g.na_lo = reinterpret_cast<uint32_t*>(a->HA + layer * a->ha_stride + (long)(F_Kt + kKtPad) * 64);
      g.na_Kt = F_Kt;
      break;
    }
    default: {  // PH_LM
      const int s = 2 * a->D;
      g.W = a->w_lm;
      g.Nt = (a->V + 15) / 16;
      g.Kt = Kt_H;
      g.Ahi = a->XA + s * a->xa_stride;
      g.Alo = g.Ahi + (long)(Kt_H + kKtPad) * 64;
      g.stats = a->XS + s * a->xs_stride;
      break;
    }
  }
  return g;
}

// A work-group's share of a GEMM phase (see gemm_phase): output range rg (n-tiles
// [t0, t0 + T), chunks of TN), K part kgi, this wave's k-tiles [k0, k1), nbr steps per
// chunk and total steps of its stream.
struct GemmGeom {
  int rg, kgi, t0, T, nch, k0, k1, nbr, total, kw_last;
};
template <int TN>
__device__ __forceinline__ GemmGeom gemm_geom(Args a, int kind, int kg, int wave) {
  constexpr int NS = gemm_ns(TN);
  GemmGeom q;
  q.kgi = blockIdx.x % kg;
  q.rg = blockIdx.x / kg;
  const int nq = a->nq[kind], nr = a->nr[kind], kq = a->kq[kind], kr = a->kr[kind];
  q.t0 = q.rg * nq + min(q.rg, nr);
  q.T = nq + (q.rg < nr ? 1 : 0);
  q.nch = (q.T + TN - 1) / TN;
  const int kb = q.kgi * kq + min(q.kgi, kr);
  const int TK = kq + (q.kgi < kr ? 1 : 0);
  // wave w takes TK / 8 k-tiles, the first TK % 8 waves one more
  const int kw = TK / kWaves, kx = TK % kWaves;
  q.k0 = kb + wave * kw + min(wave, kx);
  q.k1 = q.k0 + kw + (wave < kx ? 1 : 0);
  // steps per chunk: the longest slice rounded up to a multiple of NS (the same for every
  // wave, so that all waves reach each chunk end together)
  const int slice = kw + (kx > 0 ? 1 : 0);
  q.nbr = max(NS, ((slice + NS - 1) / NS) * NS);
  q.total = q.T > 0 ? q.nch * q.nbr : 0;
  q.kw_last = max(q.k1 - 1, 0);
  return q;
}

// One GEMM phase, y = x W^T for the 16 block rows.  The work-groups form R = blocks / kg
// output ranges of consecutive n-tiles (sizes differ by at most one tile), kg work-groups
// per range, work-group k of a range taking the k-th of kg near-equal parts of the K
// range.  A work-group walks its n-tiles in chunks of TN; its 8 waves split its K part
// into 8 contiguous slices, and a wave accumulates all TN tiles of a chunk over its slice,
// so each A fragment it loads serves TN weight tiles.  Loads form one stream per wave,
// one k-tile (TN weight tiles and the hi/lo A fragments) per step, NS steps in flight in
// NS register sets that rotate; slices are padded to a multiple of NS steps with zero A
// fragments (the weight loads of padding steps re-read a real tile).  The loop body has
// no conditional loads, so the compiler's memory wait counts stay exact.  At the end of a
// chunk the waves' sums meet in LDS and are added in wave order; with kg = 1 wave j then
// finishes tile j of the chunk, otherwise the work-groups but the range's first store their
// partial tiles (tagged, see the split-K combine below) and the first adds the kg partials in
// K order and finishes the range's tiles, so results never depend on timing.  The first NS
// steps of weights are requested before the grid barrier: they do not depend on the previous
// phase.
template <int EPI, int TN>
__device__ __forceinline__ void gemm_phase(Args a, Call c, const GemmJob& g, int kind, int kg, const PhaseCtl& pc,
                                           Failed failed, u32x4* smem) {
  constexpr int NS = gemm_ns(TN);
  static_assert(TN <= kTNMax && TN <= kWaves, "one tile per wave in the chunk epilogue");
  f32x4* red = reinterpret_cast<f32x4*>(smem);
  float* s_rstd = reinterpret_cast<float*>(reinterpret_cast<char*>(smem) + kLdsRedBytes);
  float* s_bv = s_rstd + 16;                        // ARGMAX: [TN][16]
  int* s_bi = reinterpret_cast<int*>(s_bv + kTNMax * 16);
  int* s_flag = s_bi + kTNMax * 16;

  // every lane-dependent value of a phase derives from a laundered thread index, so that the
  // compiler cannot hoist it out of the phase loop and keep it in registers for all phases
  const int tid = opaque(threadIdx.x), lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nblk = gridDim.x, b = blockIdx.x;
  const GemmGeom geo = gemm_geom<TN>(a, kind, kg, wave);
  const int rg = geo.rg, t0 = geo.t0, T = geo.T, nch = geo.nch, k0 = geo.k0, k1 = geo.k1, nbr = geo.nbr,
            total = geo.total;
  const int M = a->B;

  const GLOBAL u32x4* Wg = gbl(g.W) + lane;
  const GLOBAL u32x4* Ah = gbl(g.Ahi) + lane;
  const GLOBAL u32x4* Al = gbl(g.Alo) + lane;
  const GLOBAL u32x4* Zt = gbl(a->zero) + lane;

  // Load cursor: the NS steps of a block share their chunk (nbr is a multiple of NS), so the
  // tile offsets wb[j] of a chunk are recomputed only when a block starts a new chunk.
  long wb[TN];
  auto chunk_bases = [&](int ch) {
    const int tl = min(TN, T - ch * TN) - 1;  // last real tile of the chunk
#pragma unroll
    for (int j = 0; j < TN; ++j) wb[j] = (long)(t0 + ch * TN + min(j, tl)) * g.Kt * 64;
  };
  // the weight tiles and A fragments of step kb + i of the current chunk; padding steps past
  // the wave's slice re-read its last tile with zero A fragments
  auto load_step = [&](u32x4* w, u32x4& hv, u32x4& lv, int kb, int i) {
    const int k = k0 + kb + i;
    const long ko = (long)min(k, geo.kw_last) * 64;
#pragma unroll
    for (int j = 0; j < TN; ++j) w[j] = __builtin_nontemporal_load(Wg + wb[j] + ko);
    const bool real = k < k1;
    hv = *(real ? Ah + (long)k * 64 : Zt);
    lv = *(real ? Al + (long)k * 64 : Zt);
  };

  float best_v = -INFINITY;  // ARGMAX: running best of the work-group per row (threads < 16)
  int best_i = 0x7FFFFFFF;

  // The first NS steps' weights go out before the grid barrier (they do not depend on the
  // previous phase), their A fragments after it.
  u32x4 w[NS][TN], ah[NS], al[NS];
  auto first_weights = [&]() {
    chunk_bases(0);
#pragma unroll
    for (int i = 0; i < NS; ++i) {
      const long ko = (long)min(k0 + i, geo.kw_last) * 64;
#pragma unroll
      for (int j = 0; j < TN; ++j) w[i][j] = __builtin_nontemporal_load(Wg + wb[j] + ko);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  if (total > 0) first_weights();
  phase_begin(a, c, pc, failed);
  if (total > 0) {
#pragma unroll
    for (int i = 0; i < NS; ++i) {
      const int k = k0 + i;
      ah[i] = *(k < k1 ? Ah + (long)k * 64 : Zt);
      al[i] = *(k < k1 ? Al + (long)k * 64 : Zt);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  // sums of squares of the RMSNorm input: thread (row, part) = (tid / 32, tid % 32) sums
  // tiles part, part+32, ...; loads unconditional with clamped indices, so that no branch
  // precedes the loop; values past the last tile are dropped when summed.
  const int n_st = a->H / 16;
  float stv[8];
  if (g.stats) {
    const int row = tid >> 5, part = tid & 31;
#pragma unroll
    for (int qq = 0; qq < 8; ++qq) stv[qq] = gbl(g.stats)[min(part + 32 * qq, n_st - 1) * kStatsPad + row];
  }
  __builtin_amdgcn_sched_barrier(0);

  f32x4 acc[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};

  f32x4 own = f32x4{0.f, 0.f, 0.f, 0.f};  // split K: the reducer's own partial of tile `wave`
  EpiIn ein{};                             // epilogue inputs of the tile this wave finishes
  // end of chunk ch: the waves' partial sums meet in LDS; wave j finishes tile j
  auto chunk_end = [&](int ch) {
    if (wave < min(TN, T - ch * TN) && (kg == 1 || geo.kgi == 0))
      ein = epilogue_inputs<EPI>(a, c, g, t0 + ch * TN + wave);
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      red[(wave * TN + j) * 64 + lane] = acc[j];
      acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    if (ch == 0 && g.stats) {  // 1/rms of the rows: (x*g/rms) W^T = (1/rms) (x*g) W^T
      const int row = tid >> 5;
      float s = 0.f;
#pragma unroll
      for (int q = 0; q < 8; ++q) s += ((tid & 31) + 32 * q < n_st) ? stv[q] : 0.f;
      for (int t = (tid & 31) + 256; t < n_st; t += 32) s += gbl(g.stats)[t * kStatsPad + row];
      s += __shfl_xor(s, 16);
      s += __shfl_xor(s, 8);
      s += __shfl_xor(s, 4);
      s += __shfl_xor(s, 2);
      s += __shfl_xor(s, 1);
      if ((tid & 31) == 0) s_rstd[row] = (row < M) ? rsqrtf(s / a->H + a->eps) : 0.f;
    }
    __syncthreads();
    const int tn_c = min(TN, T - ch * TN);
    if (wave < tn_c) {
      const f32x4* rp = red + wave * 64 + lane;
      f32x4 v = rp[0];
#pragma unroll
      for (int q = 1; q < kWaves; ++q) v += rp[q * TN * 64];
      if (g.stats) {
        const int quad = (opaque(threadIdx.x) & 63) >> 4;
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] *= s_rstd[quad * 4 + i];
      }
      if (kg > 1) {
        // the partial, its low mantissa bits replaced by this use's tag (2^-23 relative)
        u32x4 t = __builtin_bit_cast(u32x4, v);
#pragma unroll
        for (int e = 0; e < 4; ++e) t[e] = (t[e] & ~1u) | g.tag;
        if (geo.kgi == 0) own = __builtin_bit_cast(f32x4, t);
        else st_wt16(reinterpret_cast<f32x4*>(g.part) + (((long)b * kTNMax + wave) * 64 + lane), t);
      } else {
        gemm_epilogue<EPI>(a, c, g, t0 + ch * TN + wave, v, ein, wave, s_bv, s_bi);
      }
    }
    if constexpr (EPI == EPI_ARGMAX) {
      __syncthreads();
      if (tid < 16)
        for (int j = 0; j < tn_c; ++j) {  // tile order: ties keep the lowest token id
          const float ov = s_bv[j * 16 + tid];
          const int oi = s_bi[j * 16 + tid];
          if (ov > best_v || (ov == best_v && oi < best_i)) {
            best_v = ov;
            best_i = oi;
          }
        }
    }
    __syncthreads();  // LDS is reused by the next chunk
  };

  // The scheduling barriers keep each set's reload right after its MFMAs: left alone, the
  // compiler sinks a reload past the other sets' MFMAs, and the wait for the next set then
  // drains every load in flight.  The last NS steps (total is a multiple of NS) request
  // nothing more.
  int lch = 0, lkb = 0;  // chunk and first step of the block being requested
  int cch = 0, ckb = 0;  // chunk and first step of the block being consumed
  for (int s0 = 0; s0 + NS < total; s0 += NS) {
    lkb += NS;
    if (lkb == nbr) {
      lkb = 0;
      ++lch;
      chunk_bases(lch);
    }
#pragma unroll
    for (int i = 0; i < NS; ++i) {
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        acc[j] = mfma(ah[i], w[i][j], acc[j]);
        acc[j] = mfma(al[i], w[i][j], acc[j]);
      }
      __builtin_amdgcn_sched_barrier(0);
      load_step(w[i], ah[i], al[i], lkb, i);
      __builtin_amdgcn_sched_barrier(0);
    }
    ckb += NS;
    if (ckb == nbr) {
      ckb = 0;
      chunk_end(cch++);
    }
  }
  if (total > 0) {
#pragma unroll
    for (int i = 0; i < NS; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        acc[j] = mfma(ah[i], w[i][j], acc[j]);
        acc[j] = mfma(al[i], w[i][j], acc[j]);
      }
    trace_mark(c, pc.slot + 1, pc.nslots);
    chunk_end(nch - 1);
    trace_mark(c, pc.slot + 2, pc.nslots);
  }

  if (kg > 1 && total > 0 && geo.kgi == 0 && wave < T) {
    // split K: work-group 0 of the range adds the kg partials of its tiles in K order.  Every
    // partial word carries the tag of this use of the partial area (the area of a phase kind
    // is used once per layer, and the tag alternates between uses), so a load that returns
    // the tag returns this use's value: the other work-groups store and go on, and the
    // reducer polls their partials directly, with no counter in between.
    const f32x4* pp = reinterpret_cast<const f32x4*>(g.part) + (((long)rg * kg * kTNMax + wave) * 64 + lane);
    f32x4 pq[kMaxSplit];
    const long long tw = wall_clock64();
    while (true) {
      bool ok = true;
#pragma unroll
      for (int q = 1; q < kMaxSplit; ++q)
        if (q < kg) {
          pq[q] = ld_coh16(pp + (long)q * kTNMax * 64);
          const u32x4 t = __builtin_bit_cast(u32x4, pq[q]);
          ok = ok && ((t[0] & t[1] & t[2] & t[3] & 1u) == g.tag) && (((t[0] | t[1] | t[2] | t[3]) & 1u) == g.tag);
        }
      if (__all(ok)) break;
      __builtin_amdgcn_s_sleep(1);
      if (wall_clock64() - tw > kBarrierTimeout) {
        if (lane == 0) __hip_atomic_store(a->err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        break;
      }
    }
    f32x4 v = own;
#pragma unroll
    for (int q = 1; q < kMaxSplit; ++q)
      if (q < kg) v += pq[q];
    gemm_epilogue<EPI>(a, c, g, t0 + wave, v, ein, wave, s_bv, s_bi);
  }

  if constexpr (EPI == EPI_ARGMAX) {
    // The work-group's best per row; the last work-group to finish picks across all of them.
    if (tid < 16) {
      st_wt(a->pmax + b * kStatsPad + tid, best_v);
      st_wt(a->pidx + b * kStatsPad + tid, best_i);
    }
    wait_vm();
    __syncthreads();
    if (tid == 0) {
      const unsigned old = __hip_atomic_fetch_add(a->done, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      *s_flag = (old == (c->done_epoch + 1u) * (unsigned)nblk - 1u) ? 1 : 0;
    }
    __syncthreads();
    if (*s_flag)  // wave w reduces rows w, w + 8 over the work-groups
      for (int row = wave; row < M; row += kWaves) {
        float v = -INFINITY;
        int ix = 0x7FFFFFFF;
        for (int w2 = lane; w2 < nblk; w2 += 64) {
          const float ov = ld_coh(a->pmax + w2 * kStatsPad + row);
          const int oi = ld_coh(a->pidx + w2 * kStatsPad + row);
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
        if (lane == 0) c->tokens[row] = (ix == 0x7FFFFFFF) ? 0 : ix;
      }
  }
}

// ---- ATTN + COMB: block attention split over the key axis, and the merge of the splits ----
// Sec. 3.2: no mask; every block row attends to the whole context and the whole block.
//
// Work item (chunk c, KV head g): context keys [c*CK, c*CK + CK); the last chunk holds keys
// [c*CK, L + B): its context tail, then the B block keys (cache slots L .. L+B-1, written by
// the QKV phase).  Rows of an item: the G query heads of g times 16 block positions (row
// t*16 + b is query head g*G + t at position b; rows b >= B are zero queries, dropped).
// K rows and V^T rows of the item (fp16) sit in the LDS staging area in 16-byte pieces with
// XOR-swizzled columns (kswz, vswz: the eight lanes of every 16-byte LDS access read eight
// different 16-byte bank groups).  The context pieces are streamed in ahead, in an earlier
// phase, by waves that issue no other loads there; pieces that hold slot L or later (K rows of the block keys and beyond, V^T lines of
// 64 keys that reach slot L) are not fetched then, because the QKV phase writes them (a cache
// line is read in a launch only after its last write there), and are loaded after it.
// Wave w takes query head t = w % G against part w / G of the item's 32-key blocks.  Scores
// are formed transposed, S^T = K Q^T, so that the probabilities land in the B-operand layout
// of the P V product and never leave registers: the A rows of the two 16-key score tiles of
// a block are keys 8*(i/4) + (i%4) and 8*(i/4) + 4 + (i%4), so lane group qd ends up holding
// keys 8 qd .. 8 qd + 7, one 16-byte V^T piece per lane for the P V product.  Queries and
// probabilities enter the fp16 matrix cores as hi/lo pairs (about 22 significant bits).  The
// parts meet in LDS, and the item's partial (running max and sum in the log2 domain, output
// divided by the sum, in fp16) is stored.
// COMB: once every item of KV head g is stored (one counter per KV head in the persistent
// launch, instead of a grid barrier), the work-groups that held them merge the chunks, each
// a share of the rows, and write the A fragments of the output projection.
template <int HD>
struct AttnShape {
  static constexpr int CK = HD == 64 ? 256 : 128;  // context keys per chunk
  static constexpr int CKM = CK + 32;              // key slots held (room for the B <= 16 block keys)
  static constexpr int NKB = CKM / 32;             // 32-key blocks
  static constexpr int KC = HD / 8;                // 16-byte pieces of a K row
  static constexpr int VC = CKM / 8;               // 16-byte pieces of a V^T row (a multiple of 4)
  static constexpr int KP = CKM * KC, VP = HD * VC;
  static constexpr int KB = KP / 64, VB = VP / 64;  // 1 KiB staging blocks
  static_assert(KP % 64 == 0 && VP % 64 == 0, "whole staging blocks");
  static_assert(kStageOff + (KP + VP) * 16 <= kLdsBytes, "LDS staging");
};

__device__ __forceinline__ int attn_chunks(int L, int CK) { return L > 0 ? (L + CK - 1) / CK : 1; }
// LDS column swizzles of the staging area: K row r, V^T row d
__device__ __forceinline__ int kswz(int r) { return (r & 3) | ((r >> 1) & 4); }
__device__ __forceinline__ int vswz(int d) { return (d >> 1) & 3; }

// Stream the context pieces of attention item j of `layer` into the LDS staging area with
// LDS-direct loads, by waves w0 .. 7: one instruction fills 64 consecutive staging slots
// (1 KiB), lane l fetching the piece that belongs in slot l, so the swizzled layout comes
// for free.  Slots whose piece is not fetched early get the cache's first piece.
template <int HD>
__device__ __forceinline__ void attn_stage(Args a, Call dc, int layer, int j, u32x4* smem, int w0) {
  using A = AttnShape<HD>;
  const int L = ctx_len(dc), nkv = a->n_kv;
  const int wave = __builtin_amdgcn_readfirstlane(opaque(threadIdx.x) >> 6);
  if (wave < w0 || j >= attn_chunks(L, A::CK) * nkv) return;
  const int c = j / nkv, g = j - (j / nkv) * nkv;
  const int kbeg = c * A::CK, Lcap = a->Lcap;
  const uint16_t* kc = a->kc + layer * a->cache_layer + (long)g * Lcap * HD + (long)kbeg * HD;
  const uint16_t* vt = a->vt + layer * a->cache_layer + (long)g * HD * Lcap + kbeg;
  const int lane = opaque(threadIdx.x) & 63;
  constexpr int RPB = 64 / A::KC;  // K rows per staging block
  const int lr = lane / A::KC, lcol = lane % A::KC;
  const int ctx = L - kbeg;        // item-relative slots below ctx are context
  LDSP char* stage = (LDSP char*)(char*)smem + kStageOff;
  for (int bl = wave - w0; bl < A::KB + A::VB; bl += kWaves - w0) {
    const uint16_t* src;
    if (bl < A::KB) {
      const int r = bl * RPB + lr;
      src = r < ctx ? kc + r * HD + ((lcol ^ kswz(r)) << 3) : a->kc;
    } else {
      const int p = (bl - A::KB) * 64 + lane;
      const int d = p / A::VC;
      const int col = (p - d * A::VC) ^ vswz(d);
      // a V^T line (64 keys) is fetched early only if all its keys are context
      const int line_end = ((kbeg + col * 8) & ~63) + 64 - kbeg;
      src = line_end <= ctx ? vt + d * Lcap + col * 8 : a->kc;
    }
    __builtin_amdgcn_global_load_lds(src, stage + bl * 1024, 16, 0, 0);
  }
}

template <int HD>
__device__ __forceinline__ void phase_attn(Args a, Call dc, int layer, const PhaseCtl& pc, Failed failed,
                                           u32x4* smem, bool staged) {
  using A = AttnShape<HD>;
  constexpr int CK = A::CK, NKB = A::NKB, KC = A::KC, VC = A::VC, KP = A::KP;
  constexpr int DT = HD / 16;  // 16-dim tiles of an output row
  static_assert(KC >= 8, "K swizzle needs 8 columns");
  u32x4* sK = smem + kStageOff / 16;                               // (row r, col) at r*KC + (col ^ kswz(r))
  u32x4* sV = sK + KP;                                             // (row d, col) at d*VC + (col ^ vswz(d))
  f32x4* sO = reinterpret_cast<f32x4*>(smem);                      // merge: [kWaves][DT][64]
  float2* sML = reinterpret_cast<float2*>(sO + kWaves * DT * 64);  // [kWaves][16]
  static_assert(kWaves * DT * 64 * 16 + kWaves * 16 * 8 <= kFailOff, "LDS merge area");

  const int L = ctx_len(dc), B = a->B, nkv = a->n_kv, G = a->n_q / a->n_kv, Lcap = a->Lcap;
  const int nch = attn_chunks(L, CK);
  const int items = nch * nkv;
  const int KS = kWaves / G;  // key parts
  const int tid = opaque(threadIdx.x), lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int t = w % G, kh = w / G;
  const bool active = kh < KS;
  const int q = lane & 15, qd = lane >> 4;
  const float* Qg = a->Q + layer * a->q_stride;
  const int q_dim = a->n_q * HD;

  // one item: everything after its context pieces are in LDS (or, without staging, all of it)
  auto item = [&](int j, bool ctx_staged) {
    const int c = j / nkv, g = j - (j / nkv) * nkv;
    const int kbeg = c * CK;
    const bool last = c == nch - 1;
    const int nkeys = last ? L + B - kbeg : CK;
    const uint16_t* kc = a->kc + layer * a->cache_layer + (long)g * Lcap * HD + (long)kbeg * HD;
    const uint16_t* vt = a->vt + layer * a->cache_layer + (long)g * HD * Lcap + kbeg;
    // queries of this wave's head: lane (row q, dims 8 qd .. 8 qd + 7 of each 32-dim slice)
    u32x4 qx[HD / 16];
    {
      const float* src = Qg + q * q_dim + (g * G + t) * HD + qd * 8;
#pragma unroll
      for (int ks = 0; ks < HD / 32; ++ks) {
        qx[2 * ks] = *gbl(reinterpret_cast<const u32x4*>(src + ks * 32));
        qx[2 * ks + 1] = *gbl(reinterpret_cast<const u32x4*>(src + ks * 32 + 4));
      }
    }
    // pieces still missing: without staging every piece of the item's keys; with staging those
    // holding slot L or later (only the last chunk has them)
    if (!ctx_staged) {
      const int nkr = min(nkeys, A::CKM);
      for (int p = tid; p < nkr * KC; p += kThreads) {
        const int r = p / KC, col = p % KC;
        sK[r * KC + (col ^ kswz(r))] = *gbl(reinterpret_cast<const u32x4*>(kc + r * HD + col * 8));
      }
      // V^T pieces of every 32-key block that is processed (keys past the end must be finite)
      const int nvc = ((nkeys + 31) >> 5) * 4;
      for (int p = tid; p < HD * nvc; p += kThreads) {
        const int d = p / nvc, col = p - (p / nvc) * nvc;
        sV[d * VC + (col ^ vswz(d))] = *gbl(reinterpret_cast<const u32x4*>(vt + d * Lcap + col * 8));
      }
    } else if (last) {
      const int rL = L - kbeg;  // first block row
      for (int p = tid; p < B * KC; p += kThreads) {
        const int r = rL + p / KC, col = p % KC;
        sK[r * KC + (col ^ kswz(r))] = *gbl(reinterpret_cast<const u32x4*>(kc + r * HD + col * 8));
      }
      // V^T pieces of the 64-key lines that reach slot L, inside the item's window
      const int c0 = (((L & ~63) - kbeg) >> 3) > 0 ? ((L & ~63) - kbeg) >> 3 : 0;
      const int c1 = min(VC, (((L + B + 63) & ~63) - kbeg) >> 3);
      const int nv = c1 - c0;
      for (int p = tid; p < HD * nv; p += kThreads) {
        const int d = p / nv, col = c0 + p - (p / nv) * nv;
        sV[d * VC + (col ^ vswz(d))] = *gbl(reinterpret_cast<const u32x4*>(vt + d * Lcap + col * 8));
      }
    }
    __syncthreads();
    if (j == (int)blockIdx.x) trace_mark(dc, pc.slot + 1, pc.nslots);

    // this wave's 32-key blocks [kb0, kb1)
    const int nkb = (nkeys + 31) >> 5, bps = (nkb + KS - 1) / KS;
    const int kb0 = min(kh * bps, nkb), kb1 = min(kb0 + bps, nkb);
    float m = -INFINITY, l = 0.f;
    f32x4 o[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (active && kb1 > kb0) {
      u32x4 qh[HD / 32], ql[HD / 32];
#pragma unroll
      for (int ks = 0; ks < HD / 32; ++ks) {
        const float s = a->qscale;
        const u32x4 x0 = qx[2 * ks], x1 = qx[2 * ks + 1];
        float v[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[e] = __uint_as_float(x0[e]) * s;
          v[4 + e] = __uint_as_float(x1[e]) * s;
        }
        split_pack8_h(v, qh[ks], ql[ks]);
      }
      // LDS read addresses: per-lane byte bases plus compile-time offsets.  Score tile kt of a
      // block reads K row 8*(q/4) + 4*kt + (q%4) (its swizzle is kswz of that row, the same for
      // every block and tile); V^T row d = dt*16 + q has swizzle vswz(q).
      const char* lds = reinterpret_cast<const char*>(smem);
      const int kr = 8 * (q >> 2) + (q & 3), ksw = kswz(kr);
      int k_at[HD / 32];
#pragma unroll
      for (int ks = 0; ks < HD / 32; ++ks) k_at[ks] = opaque(kStageOff + (kr * KC + ((ks * 4 + qd) ^ ksw)) * 16);
      const int v_at = opaque(kStageOff + KP * 16 + (q * VC + (qd ^ vswz(q))) * 16);
      // scores of the wave's blocks; other blocks and keys past the end: -inf
      f32x4 sc[2 * NKB];
#pragma unroll
      for (int kk = 0; kk < NKB; ++kk) {
        f32x4 a0 = {-INFINITY, -INFINITY, -INFINITY, -INFINITY}, a1 = a0;
        if (kk >= kb0 && kk < kb1) {
          f32x4 h0 = {0.f, 0.f, 0.f, 0.f}, l0 = h0, h1 = h0, l1 = h0;
          u32x4 k0v[HD / 32], k1v[HD / 32];
#pragma unroll
          for (int ks = 0; ks < HD / 32; ++ks) {
            k0v[ks] = *reinterpret_cast<const u32x4*>(lds + k_at[ks] + (kk * 32) * KC * 16);
            k1v[ks] = *reinterpret_cast<const u32x4*>(lds + k_at[ks] + (kk * 32 + 4) * KC * 16);
          }
#pragma unroll
          for (int ks = 0; ks < HD / 32; ++ks) {
            h0 = mfma_h(k0v[ks], qh[ks], h0);
            h1 = mfma_h(k1v[ks], qh[ks], h1);
            l0 = mfma_h(k0v[ks], ql[ks], l0);
            l1 = mfma_h(k1v[ks], ql[ks], l1);
          }
          a0 = h0 + l0;
          a1 = h1 + l1;
          if ((kk + 1) * 32 > nkeys) {  // the block reaches past the item's keys
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              if (kk * 32 + qd * 8 + i >= nkeys) a0[i] = -INFINITY;
              if (kk * 32 + qd * 8 + 4 + i >= nkeys) a1[i] = -INFINITY;
            }
          }
        }
        sc[2 * kk] = a0;
        sc[2 * kk + 1] = a1;
      }
      // softmax statistics per query row (column q), in the log2 domain
#pragma unroll
      for (int kt = 0; kt < 2 * NKB; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) m = fmaxf(m, sc[kt][i]);
      m = fmaxf(m, __shfl_xor(m, 16));
      m = fmaxf(m, __shfl_xor(m, 32));
#pragma unroll
      for (int kk = 0; kk < NKB; ++kk) {
        if (kk >= kb0 && kk < kb1) {  // the other blocks' probabilities are never used
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float p = __builtin_amdgcn_exp2f(sc[2 * kk + h][i] - m);
              sc[2 * kk + h][i] = p;
              l += p;
            }
        }
      }
      l += __shfl_xor(l, 16);
      l += __shfl_xor(l, 32);
      // O^T = V^T P^T over the wave's blocks
#pragma unroll
      for (int kk = 0; kk < NKB; ++kk) {
        if (kk >= kb0 && kk < kb1) {
          float pv[8] = {sc[2 * kk][0], sc[2 * kk][1], sc[2 * kk][2], sc[2 * kk][3],
                         sc[2 * kk + 1][0], sc[2 * kk + 1][1], sc[2 * kk + 1][2], sc[2 * kk + 1][3]};
          u32x4 ph, pl;
          split_pack8_hz(pv, ph, pl);
          // keys kk*32 + 8*qd .. + 7: the 16-byte V^T piece kk*4 + qd of row dt*16 + q
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            const u32x4 vv = *reinterpret_cast<const u32x4*>(lds + v_at + (dt * 16 * VC + kk * 4) * 16);
            o[dt] = mfma_h(vv, ph, o[dt]);
            o[dt] = mfma_h(vv, pl, o[dt]);
          }
        }
      }
    }
    if (j == (int)blockIdx.x && w == 0) trace_mark(dc, pc.slot + 2, pc.nslots);
    // merge the key parts of each head (part order), then store the item's partial
    if (KS > 1) {
      if (active && kh > 0) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) sO[(w * DT + dt) * 64 + lane] = o[dt];
        if (qd == 0) sML[w * 16 + q] = make_float2(m, l);
      }
      __syncthreads();
      if (kh == 0) {
        for (int k = 1; k < KS; ++k) {
          const int wk = t + k * G;
          const float2 mlk = sML[wk * 16 + q];
          const float M = fmaxf(m, mlk.x);
          const float f0 = __builtin_amdgcn_exp2f(m - M), f1 = __builtin_amdgcn_exp2f(mlk.x - M);  // 0 for a part without keys
          l = f0 * l + f1 * mlk.y;
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) o[dt] = f0 * o[dt] + f1 * sO[(wk * DT + dt) * 64 + lane];
          m = M;
        }
      }
    }
    if (kh == 0 && q < B) {
      const long row = ((long)layer * a->nch * nkv + (long)c * nkv + g) * (G * 16) + t * 16 + q;
      uint16_t* op = a->OP + row * HD + qd * 4;
      const float inv = 1.0f / l;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const uint64_t hv = (uint64_t)f2h(o[dt][0] * inv) | ((uint64_t)f2h(o[dt][1] * inv) << 16) |
                            ((uint64_t)f2h(o[dt][2] * inv) << 32) | ((uint64_t)f2h(o[dt][3] * inv) << 48);
        st_wt8(op + dt * 16, hv);
      }
      if (qd == 0) st_wt8(a->ML + row, (uint64_t)__float_as_uint(m) | ((uint64_t)__float_as_uint(l) << 32));
    }
    // the item is stored: count it for its KV head
    wait_vm();
    __syncthreads();
    // (chunk 0 also adds the chunks this context does not have, so that every layer adds
    // a->nch per KV head whatever the context length, and the host's count needs no length)
    if (tid == 0)
      __hip_atomic_fetch_add(a->acnt + g * 32, c == 0 ? 1u + (unsigned)(a->nch - nch) : 1u, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
  };

  // One call site for the item body keeps the phase's code small.
  // no grid barrier before this phase: each item waits for its KV head's Q/K/V tiles
  if (!pc.wait || (int)blockIdx.x >= items) trace_mark(dc, pc.slot, pc.nslots);
  for (int j = blockIdx.x; j < items; j += gridDim.x) {
    if (pc.wait) {
      qkv_wait(a, dc, layer, j % nkv, failed);
      if (j == (int)blockIdx.x) trace_mark(dc, pc.slot, pc.nslots);
    }
    item(j, staged && j == (int)blockIdx.x);
  }
}

// COMB: work-groups b < W * n_kv (W = work-groups per KV head) merge the chunks of KV head
// g = b % n_kv for a share of its G*B rows, on waves 0-3: a row's chunks are split into S
// runs over S waves (S = 4 / rows per work-group), which meet in LDS in run order.  Waves
// 4-7 meanwhile stream the context of the next layer's attention item into LDS (stage).
template <int HD>
__device__ __forceinline__ void phase_comb(Args a, Call dc, int layer, const PhaseCtl& pc, Failed failed, u32x4* smem,
                           bool stage) {
  using A = AttnShape<HD>;
  constexpr int DPL = HD / 64;                 // dims per lane
  constexpr int CB = DPL == 2 ? 16 : 32;       // chunks whose loads are in flight together
  constexpr int CW = 4;                        // waves that merge
  const int L = ctx_len(dc), B = a->B, nkv = a->n_kv, G = a->n_q / a->n_kv;
  const int nch = attn_chunks(L, A::CK);
  const int W = min(nch, (int)gridDim.x / nkv);
  const int b = blockIdx.x;
  if (stage) attn_stage<HD>(a, dc, layer + 1, b, smem, CW);
  // the group wait: all items of KV head g stored (persistent launch; else the launch boundary)
  if (pc.wait) {
    if (b < W * nkv && threadIdx.x < 64 && !*failed) {
      const unsigned* cnt = a->acnt + (b % nkv) * 32;
      const unsigned target = dc->acnt_base + (unsigned)(layer + 1) * (unsigned)a->nch;
      const long long t0 = wall_clock64();
      while (__hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
        __builtin_amdgcn_s_sleep(1);
        if (wall_clock64() - t0 > kBarrierTimeout) {
          if (threadIdx.x == 0) {
            *failed = 1;
            __hip_atomic_store(a->err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
          }
          break;
        }
      }
    }
    __syncthreads();
  }
  trace_mark(dc, pc.slot, pc.nslots);
  if (b >= W * nkv) return;
  const int g = b % nkv, wi = b / nkv;
  const int nrows = G * B;
  const int rpw = (nrows + W - 1) / W;                 // rows of this work-group
  const int r0 = wi * rpw, r1 = min(nrows, r0 + rpw);
  const int S = rpw >= CW ? 1 : CW / rpw;              // runs per row
  const int cps = (nch + S - 1) / S;                   // chunks per run
  const int lane = opaque(threadIdx.x) & 63;
  const int w = __builtin_amdgcn_readfirstlane(opaque(threadIdx.x) >> 6);
  float* sN = reinterpret_cast<float*>(smem);          // [CW][64][DPL] run numerators
  float2* sMD = reinterpret_cast<float2*>(sN + CW * 64 * DPL);  // [CW] run (max, denominator)
  const int q_Kt = a->n_q * HD / 32;
  uint32_t* ohi = reinterpret_cast<uint32_t*>(a->OA + layer * a->oa_stride);
  uint32_t* olo = reinterpret_cast<uint32_t*>(a->OA + layer * a->oa_stride + (long)(q_Kt + kKtPad) * 64);
  const long cstride = (long)nkv * G * 16;  // rows between chunks
  const long lbase = (long)layer * a->nch * cstride + (long)g * G * 16;
  // rounds of (row, run) units: unit u = w + CW k -> row r0 + u / S, run u % S
  const int units = (r1 - r0) * S;
  for (int u0 = 0; u0 < units; u0 += CW) {
    const int u = u0 + w;
    const bool has = w < CW && u < units;
    const int rr = r0 + (has ? u / S : 0), run = has ? u % S : 0;
    const int tt = rr / B, bb = rr - (rr / B) * B;
    const long row = lbase + tt * 16 + bb;
    const int cb = run * cps, ce = has ? min(nch, cb + cps) : cb;
    float M = -INFINITY, den = 0.f, num[DPL];
#pragma unroll
    for (int e = 0; e < DPL; ++e) num[e] = 0.f;
    for (int c0 = cb; c0 < ce; c0 += CB) {
      float2 mc[CB];
      float ov[CB][DPL];
#pragma unroll
      for (int k = 0; k < CB; ++k) {
        const long rc = row + (long)min(c0 + k, ce - 1) * cstride;
        const uint64_t mlv = *gbl(reinterpret_cast<const uint64_t*>(a->ML + rc));
        mc[k] = make_float2(__uint_as_float((uint32_t)mlv), __uint_as_float((uint32_t)(mlv >> 32)));
        if constexpr (DPL == 2) {
          const uint32_t v = *gbl(reinterpret_cast<const uint32_t*>(a->OP + rc * HD + 2 * lane));
          ov[k][0] = h2f(v & 0xFFFFu);
          ov[k][1] = h2f(v >> 16);
        } else {
          ov[k][0] = h2f(*gbl(a->OP + rc * HD + lane));
        }
      }
      float Mb = M;
#pragma unroll
      for (int k = 0; k < CB; ++k) Mb = fmaxf(Mb, mc[k].x);
      const float f = __builtin_amdgcn_exp2f(M - Mb);  // rescale of the run so far (0 when it is empty)
      den *= f;
#pragma unroll
      for (int e = 0; e < DPL; ++e) num[e] *= f;
#pragma unroll
      for (int k = 0; k < CB; ++k) {
        if (c0 + k < ce) {
          const float wgt = __builtin_amdgcn_exp2f(mc[k].x - Mb) * mc[k].y;  // a chunk's sum times its normalised output
          den += wgt;
#pragma unroll
          for (int e = 0; e < DPL; ++e) num[e] += wgt * ov[k][e];
        }
      }
      M = Mb;
    }
    if (w == 0 && u0 == 0) trace_mark(dc, pc.slot + 1, pc.nslots);
    if (S > 1) {
      // the runs of a row meet in LDS; the wave of run 0 finishes the row
      if (w < CW) {
#pragma unroll
        for (int e = 0; e < DPL; ++e) sN[(w * 64 + lane) * DPL + e] = num[e];
        if (lane == 0) sMD[w] = make_float2(M, den);
      }
      __syncthreads();
      if (has && run == 0) {
        float Mt = M;
        for (int k = 1; k < S; ++k) Mt = fmaxf(Mt, sMD[w + k].x);
        float dt = 0.f, nt[DPL];
#pragma unroll
        for (int e = 0; e < DPL; ++e) nt[e] = 0.f;
        for (int k = 0; k < S; ++k) {
          const float2 md = sMD[w + k];
          const float f = __builtin_amdgcn_exp2f(md.x - Mt);
          dt += f * md.y;
#pragma unroll
          for (int e = 0; e < DPL; ++e) nt[e] += f * sN[((w + k) * 64 + lane) * DPL + e];
        }
        den = dt;
#pragma unroll
        for (int e = 0; e < DPL; ++e) num[e] = nt[e];
      }
      __syncthreads();
    }
    if (has && run == 0) {
      const float inv = 1.0f / den;
      const int k = (g * G + tt) * HD;
      if constexpr (DPL == 2) {
        store_frag_pair_wt(ohi, olo, bb, k + 2 * lane, q_Kt, num[0] * inv, num[1] * inv);
      } else {
        const float y = num[0] * inv;
        const float y1 = __shfl_xor(y, 1);
        if ((lane & 1) == 0) store_frag_pair_wt(ohi, olo, bb, k + lane, q_Kt, y, y1);
      }
    }
  }
}

// Chunk width of phase kind slot s (Q/K/V 0, output 1, gate/up 2, down 3) in a kernel's plan
// signature: 4 bits per slot; signature 0 leaves every width to the plan read at run time.
constexpr int sig_tn(int sig, int s) { return (sig >> (4 * s)) & 15; }

// GEMM phase with the plan's chunk width: TNF when the kernel is built for its plan, else the
// plan's width read at run time (the LM head always uses 8)
template <int EPI, int TNF>
__device__ __forceinline__ void gemm_dispatch(Args a, Call c, int kind, int layer, const PhaseCtl& pc, Failed failed,
                                              u32x4* smem) {
  GemmJob g = make_job(a, c, kind, layer);
  const int kg = kind == PH_LM ? 1 : a->kg[kind];
  const int slot = kind == PH_QKV ? 0 : kind == PH_O ? 1 : kind == PH_GU ? 2 : 3;
  g.part = a->part + (long)slot * gridDim.x * kTNMax * 256;
  g.tag = (c->done_epoch * (unsigned)a->D + (unsigned)layer + 1u) & 1u;
  if constexpr (EPI == EPI_ARGMAX) {
    gemm_phase<EPI, 8>(a, c, g, kind, 1, pc, failed, smem);
  } else if constexpr (TNF != 0) {
    gemm_phase<EPI, TNF>(a, c, g, kind, kg, pc, failed, smem);
  } else {
    switch (a->tn[kind]) {
      case 2: gemm_phase<EPI, 2>(a, c, g, kind, kg, pc, failed, smem); break;
      case 3: gemm_phase<EPI, 3>(a, c, g, kind, kg, pc, failed, smem); break;
      case 4: gemm_phase<EPI, 4>(a, c, g, kind, kg, pc, failed, smem); break;
      case 5: gemm_phase<EPI, 5>(a, c, g, kind, kg, pc, failed, smem); break;
      case 6: gemm_phase<EPI, 6>(a, c, g, kind, kg, pc, failed, smem); break;
      default: gemm_phase<EPI, 8>(a, c, g, kind, kg, pc, failed, smem); break;
    }
  }
}

// The single kernel argument is read in place through the kernel-argument pointer, so each
// field is loaded where it is used instead of being held in scalar registers (or copied to
// scratch memory, as a by-reference use of a parameter would) for the whole launch.
//
// SIG != 0 builds the kernel for one set of GEMM plans (chunk widths per phase kind, see
// sig_tn): only those GEMM bodies are instantiated, ~90 KiB of code instead of ~320 KiB.  The
// phases of a layer then run from a smaller code footprint (each phase's epilogue runs once
// per layer, so its instructions are fetched anew every layer); results are the same as the
// generic kernel's (SIG = 0), which serves every other plan.
template <int HD, int SIG>
__global__ __launch_bounds__(kThreads) void k_draft(DraftKernArgs) {
  __shared__ u32x4 smem[kLdsBytes / 16];
  const CONSTANT DraftKernArgs* ka = (const CONSTANT DraftKernArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  const Args a = (const CONSTANT DraftArgs*)ka->a;
  const Call c = &ka->c;
  const int p0 = ka->p0, p1 = ka->p1;
  const int nphase = phase_count(a->D);
  const int nslots = kTraceSlots * nphase;
  const Failed failed = (Failed)((LDSP char*)(char*)smem + kFailOff);
  if (threadIdx.x == 0) *failed = 0;
  unsigned epoch = c->bar_epoch;  // grid barriers passed
  for (int p = p0; p < p1; ++p) {
    int kind, layer;
    phase_of(p, a->D, kind, layer);
    PhaseCtl pc;
    // the attention and combine phases wait for their KV head's Q/K/V tiles and attention
    // items, every other phase at a grid barrier
    pc.wait = p > p0;
    if (pc.wait && kind != PH_ATTN && kind != PH_COMB) ++epoch;
    pc.epoch = epoch;
    pc.slot = kTraceSlots * p;
    pc.nslots = nslots;
    switch (kind) {
      case PH_EMBED:  // wave 0 embeds (its threads hold every item), waves 1-7 stage layer 0's attention item
        phase_begin(a, c, pc, failed);
        if (threadIdx.x < 64) phase_embed(a, c);
        attn_stage<HD>(a, c, 0, blockIdx.x, smem, 1);
        break;
      case PH_QKV:
        gemm_dispatch<EPI_QKV, sig_tn(SIG, 0)>(a, c, kind, layer, pc, failed, smem);
        break;
      case PH_ATTN:  // staged by the embedding phase (layer 0) or the previous layer's combine phase
        phase_attn<HD>(a, c, layer, pc, failed, smem, layer == 0 ? p - 2 >= p0 : p - 5 >= p0);
        break;
      case PH_COMB:  // stages the next layer's first attention item when that phase runs in this launch
        phase_comb<HD>(a, c, layer, pc, failed, smem, layer + 1 < a->D && p + 5 < p1);
        break;
      case PH_GU:
        gemm_dispatch<EPI_SWIGLU, sig_tn(SIG, 2)>(a, c, kind, layer, pc, failed, smem);
        break;
      case PH_O:  // one call site for both residual GEMMs: one copy of each body they use
      case PH_DOWN:
        if constexpr (sig_tn(SIG, 1) == sig_tn(SIG, 3))
          gemm_dispatch<EPI_RESID, sig_tn(SIG, 1)>(a, c, kind, layer, pc, failed, smem);
        else if (kind == PH_O)
          gemm_dispatch<EPI_RESID, sig_tn(SIG, 1)>(a, c, kind, layer, pc, failed, smem);
        else
          gemm_dispatch<EPI_RESID, sig_tn(SIG, 3)>(a, c, kind, layer, pc, failed, smem);
        break;
      default:  // PH_LM
        gemm_dispatch<EPI_ARGMAX, 0>(a, c, kind, layer, pc, failed, smem);
        break;
    }
    // the Q/K/V and attention phases hand over through the per-KV-head counters (the Q/K/V
    // counts are added in every launch: the host's count of them does not depend on the mode);
    // the staging waves of the embedding phase issued loads only: they need not wait for them
    if (kind == PH_QKV) qkv_arrive(a);
    else if (p + 1 < p1 && kind != PH_ATTN) grid_arrive(a, kind != PH_EMBED || threadIdx.x < 64);
    else wait_vm();
    trace_mark(c, kTraceSlots * p + kTraceSlots - 1, nslots);
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

void launch_compose(hipStream_t s, uint16_t* out, const uint16_t* A, const uint16_t* B, int R, int O, int K) {
  hipLaunchKernelGGL(k_compose, dim3((K + 63) / 64, (R + 63) / 64), dim3(256), 0, s, out, A, B, R, O, K);
}

void launch_matvec(hipStream_t s, float* y, const uint16_t* A, const uint16_t* b, int R, int O) {
  hipLaunchKernelGGL(k_matvec, dim3(R), dim3(256), 0, s, y, A, b, O);
}

void launch_bf16_to_f32(hipStream_t s, float* dst, const uint16_t* src, long n) {
  int blocks = (int)((n + 255) / 256);
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_bf16_to_f32, dim3(blocks), dim3(256), 0, s, dst, src, n);
}

void launch_fuse(hipStream_t s, const uint16_t* hidden, int n, int ld, int S, int H, int D, const float* alpha,
                 const float* gain, float* ustats, u32x4* ua_hi, u32x4* ua_lo, int n_max, int mt_max) {
  const int pairs = ((H + 511) / 512) * n;
  const int groups = (pairs + kXcds - 1) / kXcds;
  hipLaunchKernelGGL(k_fuse, dim3(groups * kXcds * D), dim3(64), 0, s, hidden, ld, S, H, n, D, alpha, gain, ustats,
                     ua_hi, ua_lo, n_max, mt_max);
}

// Verification (Sec. 3.2): one wave.  k = the number of leading candidates j = 1.. that
// equal the target's prediction after position j - 1; the bonus is the target's
// prediction after position k.  Writes the next block (bonus, then the mask ids), the
// emitted tokens (k candidates, bonus, then -1), k (to host-visible memory or a device
// word) and, when L_next is given, the context length after the k + 1 verified rows.
__global__ __launch_bounds__(64) void k_accept(const int32_t* block_ids, const int32_t* draft, const int32_t* target,
                                               int B, int32_t* next_ids, int32_t* emitted, int32_t* k_out,
                                               const int32_t* Lp, int L_imm, int32_t* L_next) {
  const int b = threadIdx.x;
  const bool in = b < B;
  const int d = in ? draft[b] : 0;
  const int tp = (b >= 1 && b < B) ? target[b - 1] : 0;
  const unsigned long long miss = __ballot(b >= 1 && b < B && d != tp);
  const int k = miss ? __ffsll((long long)miss) - 2 : B - 1;
  const int bonus = target[k];
  const int dn = __shfl_down(d, 1);  // candidate b + 1
  if (in) {
    next_ids[b] = b == 0 ? bonus : block_ids[b];
    emitted[b] = b < k ? dn : (b == k ? bonus : -1);
  }
  if (b == 0) __hip_atomic_store(k_out, k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  if (b == 0 && L_next) *L_next = (Lp ? *Lp : L_imm) + k + 1;  // the context after the k + 1 rows
}

void launch_accept(hipStream_t s, const int32_t* block_ids, const int32_t* draft, const int32_t* target, int B,
                   int32_t* next_ids, int32_t* emitted, int32_t* k_out, const int32_t* Lp, int L_imm,
                   int32_t* L_next) {
  hipLaunchKernelGGL(k_accept, dim3(1), dim3(64), 0, s, block_ids, draft, target, B, next_ids, emitted, k_out, Lp,
                     L_imm, L_next);
}

void launch_fused_rows(hipStream_t s, const u32x4* ua_hi, const u32x4* ua_lo, const float* ustats, int n, int H,
                       int D, int n_max, int mt_max, float eps, float* out) {
  hipLaunchKernelGGL(k_fused_rows, dim3(n, D), dim3(256), 0, s, ua_hi, ua_lo, ustats, n, H, D, n_max, mt_max, eps,
                     out);
}

bool kvt_shape_supported(int nt_per_block, int waves) {
  return (nt_per_block == 1 && waves == 16) || (nt_per_block == 2 && waves == 8);
}

void launch_kvt(hipStream_t s, int nt_per_block, int waves, const KvtArgs& a, int layers, int mtiles) {
  const dim3 grid((a.Nt + nt_per_block - 1) / nt_per_block, layers, mtiles);
  if (nt_per_block == 2 && waves == 8) hipLaunchKernelGGL((k_kvt<2, 8>), grid, dim3(512), 0, s, a);
  else hipLaunchKernelGGL((k_kvt<1, 16>), grid, dim3(1024), 0, s, a);
}

// Measurement: a plain streaming read of n16 16-byte words (eight nontemporal loads in flight
// per thread, grid-stride), the HBM read ceiling the draft kernels are compared with.  The
// XOR of the data is stored only if it equals a value it cannot be made to equal by chance
// often enough to matter, so that the loads are not removed.
__global__ __launch_bounds__(256) void k_read_probe(const u32x4* __restrict__ p, long n16, uint32_t* sink) {
  uint32_t acc = 0;
  const long stride = (long)gridDim.x * 256 * 8;
  for (long i0 = (long)blockIdx.x * 256 * 8 + threadIdx.x; i0 < n16; i0 += stride) {
    u32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const long i = i0 + u * 256;
      v[u] = i < n16 ? __builtin_nontemporal_load(p + i) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
  }
  if (acc == 0x9E3779B9u) sink[0] = acc;
}

void launch_read_probe(hipStream_t s, const void* buf, long bytes, uint32_t* sink, int blocks) {
  hipLaunchKernelGGL(k_read_probe, dim3(blocks), dim3(256), 0, s, reinterpret_cast<const u32x4*>(buf), bytes / 16,
                     sink);
}

// Kernels built for one set of plans: those the plan chooser picks on 256 work-groups for the
// Qwen3-8B, Qwen3-4B and GPT-OSS-20B shapes (signature: Q/K/V | output << 4 | gate/up << 8 |
// down << 12).  Any other head size and plan runs the generic kernel.
constexpr int kSigQwen3_8B = 3 | 4 << 4 | 6 << 8 | 4 << 12;
constexpr int kSigQwen3_4B = 3 | 3 << 4 | 5 << 8 | 3 << 12;
constexpr int kSigGptOss = 5 | 3 << 4 | 3 << 8 | 3 << 12;

static const void* draft_kernel(int hd, int sig) {
  if (hd == 128 && sig == kSigQwen3_8B) return reinterpret_cast<const void*>(&k_draft<128, kSigQwen3_8B>);
  if (hd == 128 && sig == kSigQwen3_4B) return reinterpret_cast<const void*>(&k_draft<128, kSigQwen3_4B>);
  if (hd == 64 && sig == kSigGptOss) return reinterpret_cast<const void*>(&k_draft<64, kSigGptOss>);
  return hd == 64 ? reinterpret_cast<const void*>(&k_draft<64, 0>) : reinterpret_cast<const void*>(&k_draft<128, 0>);
}

bool draft_specialized(int hd, int sig) { return draft_kernel(hd, sig) != draft_kernel(hd, 0); }

hipError_t launch_draft(hipStream_t s, const DraftArgs* a_dev, const DraftCall& c, int hd, int sig, int blocks,
                        int p0, int p1, bool cooperative) {
  DraftKernArgs ka;
  ka.a = a_dev;
  ka.c = c;
  ka.p0 = p0;
  ka.p1 = p1;
  void* kargs[] = {&ka};
  const void* fn = draft_kernel(hd, sig);
  if (cooperative) return hipLaunchCooperativeKernel(fn, dim3(blocks), dim3(kThreads), kargs, 0, s);
  return hipLaunchKernel(fn, dim3(blocks), dim3(kThreads), kargs, 0, s);
}

int draft_blocks_per_cu(int hd, int sig) {
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, draft_kernel(hd, sig), kThreads, 0) != hipSuccess) return 0;
  return n;
}

}  // namespace dflare
