// luna_noncausal.hip -- non-causal LUNA attention, eq. (9) of Section 3.1.
//
// Two schedules, chosen per call by the host:
//
//  fused    (at least 192 heads and the per-head accumulators fit in registers)
//           one launch, one workgroup of four waves per head, one wave per SIMD.
//           Each wave sums its share of S and z over the head's keys in registers,
//           the four shares are added in LDS in a fixed order and turned into
//           readout fragments, and the same workgroup then streams the head's
//           queries in groups of two 16-token blocks.  S never reaches HBM; the
//           launch is bound by issue of the feature-map arithmetic, not by HBM.
//  split    (fewer heads) the three passes below, so that a head's keys and
//           queries are spread over many workgroups.
//
// The split schedule's passes, after the table build:
//
//  state    one workgroup per (head, token range).  Each wave takes 32-token steps:
//           u = K W^T on the matrix cores (A = K rows, B = W^T), so a lane holds
//           projection 16mb + r for eight tokens; psi turns each of those into L
//           operand fragments "feature (mb, l, r) x 8 tokens".  S += phi(K)^T V and
//           z += phi(K)^T 1 accumulate in fp32 matrix-core accumulators, with V read
//           transposed from LDS.  The four waves are summed in LDS in a fixed order
//           and the range's partial (S | z) is written in fp32.
//  reduce   one workgroup per head sums the partials in range order (deterministic)
//           and writes S and z as readout operand fragments in the call's dtype.
//  readout  one workgroup per (head, 256-token tile).  u^T = W Q^T puts four
//           projections of one token in each lane, so psi's outputs are directly the
//           B fragments of num^T = S^T phi(Q)^T and den = z^T phi(Q)^T; the statistics
//           stay in registers for the whole tile.  out = num * (1 / (den + eps)).
//
// Feature order.  The state pass produces rows (mb, l, i16) ("projection-block,
// channel, projection"); the readout consumes "k-order": fragment kappa, lane group
// g, slot e stands for list position p = 8 kappa + e of (mb*4 + j)*L + l, i.e.
// projection 16mb + 4g + j and channel l (zero beyond 4*MB*L).  The reduce pass
// permutes between the two.
#include "luna_device.hpp"
#include "luna_kernels.hpp"

#include <type_traits>

namespace luna {

template <typename T, int DH, int L, int MB>
struct NcCfg {
  static constexpr int KS = DH / 32;                 // k-steps over the head dimension
  static constexpr int CB = DH / 16;                 // value-column blocks
  static constexpr int NF = (4 * MB * L + 7) / 8;    // readout fragments along features
  static constexpr int DP = 16 * MB * L;             // state rows (mb, l, i16)
  static constexpr int NSEG = nseg_cap(L, kAttnSegBytes);
  static constexpr int VE = 16 / (int)sizeof(T);     // elements per 16-byte load
  static constexpr int VROW = 36;                    // V^T row length in LDS (padded, 16-B multiple for fp32)
  static constexpr int NVC = 32 * (DH / VE) / kWave; // V 16-byte chunks per lane per step
  static constexpr size_t FRAG_ELEMS = (size_t)(CB + 1) * NF * kWave * 8;
};

// ---------------------------------------------------------------------------
// state pass
// ---------------------------------------------------------------------------
template <typename T, int DH, int L, int MB>
__global__ __launch_bounds__(256, 1) void nc_state_kernel(NoncausalArgs a) {
  using C = NcCfg<T, DH, L, MB>;
  __shared__ typename PwlTab<T, L, C::NSEG>::type tab;
  __shared__ __attribute__((aligned(16))) T vt[4][DH][C::VROW];
  __shared__ float red[C::DP][DH + 1];

  const int head = blockIdx.x / a.splits;
  const int split = blockIdx.x - head * a.splits;
  const int hset = a.phi.per_head ? head % a.H : 0;
  pwl_load(tab, a.phi.tables + (size_t)hset * kTableBytes);

  const int wave = wave_id(), lane = threadIdx.x % kWave;
  const int g = lane / 16, r = lane % 16;
  const int M = a.phi.M;
  const size_t hoff = (size_t)head * a.n * DH;
  const T* K = reinterpret_cast<const T*>(a.K) + hoff;
  const T* V = reinterpret_cast<const T*>(a.V) + hoff;
  const T* W = reinterpret_cast<const T*>(a.phi.W) + (size_t)hset * M * DH;
  const float* bias = a.phi.b + (size_t)hset * M;

  // B operand of u = K W^T: column r of block mb is projection 16mb + r.
  Frag<T> wf[MB][C::KS];
  float bcol[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int p = 16 * mb + r;
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      if (p < M) load8(wf[mb][ks], W + (size_t)p * DH + 32 * ks + 8 * g);
      else wf[mb][ks].zero();
    }
    bcol[mb] = p < M ? bias[p] : 0.0f;
  }
  Frag<T> ones;
  ones.fill(1.0f);

  f32x4 accS[MB][L][C::CB];
  f32x4 accZ[MB][L];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int l = 0; l < L; ++l) {
      accZ[mb][l] = zero4();
#pragma unroll
      for (int cb = 0; cb < C::CB; ++cb) accS[mb][l][cb] = zero4();
    }

  const int t_begin = split * a.tokens_per_split;
  const int t_end = min(a.n, t_begin + a.tokens_per_split);
  const int nsteps = (t_end - t_begin + 31) / 32;
  const int iters = (nsteps + 3) / 4;

  // registers holding the next step's K fragments and V chunks
  Frag<T> kn[2][C::KS];
  i32x4 vn[C::NVC];
  auto fetch = [&](int it) {
    const int t0 = t_begin + (it * 4 + wave) * 32;
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) {
      const int t = t0 + 16 * tb + r;
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) {
        if (t < t_end) load8(kn[tb][ks], K + (size_t)t * DH + 32 * ks + 8 * g);
        else kn[tb][ks].zero();
      }
    }
#pragma unroll
    for (int q = 0; q < C::NVC; ++q) {
      const int c = lane + kWave * q;
      const int tt = c / (DH / C::VE), cg = c % (DH / C::VE);
      const int t = t0 + tt;
      if (t < t_end) vn[q] = *reinterpret_cast<const i32x4*>(V + (size_t)t * DH + cg * C::VE);
      else vn[q] = i32x4{0, 0, 0, 0};
    }
  };

  __syncthreads();
  const int tsteps = __builtin_amdgcn_readfirstlane(tab.steps);
  const float tfloor = tab.floor;

  if (iters > 0) fetch(0);
  for (int it = 0; it < iters; ++it) {
    const int t0 = t_begin + (it * 4 + wave) * 32;
    // V^T of this step into the wave's LDS slice
#pragma unroll
    for (int q = 0; q < C::NVC; ++q) {
      const int c = lane + kWave * q;
      const int tt = c / (DH / C::VE), cg = c % (DH / C::VE);
      const T* e = reinterpret_cast<const T*>(&vn[q]);
#pragma unroll
      for (int x = 0; x < C::VE; ++x) vt[wave][cg * C::VE + x][tt] = e[x];
    }
    Frag<T> kc[2][C::KS];
#pragma unroll
    for (int tb = 0; tb < 2; ++tb)
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) kc[tb][ks] = kn[tb][ks];
    if (it + 1 < iters) fetch(it + 1);
    __syncthreads();

    // projections and channel functions -> A fragments phi(K)^T
    float uu[8 * MB];  // [mb][tb][j]
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        f32x4 acc = zero4();
#pragma unroll
        for (int ks = 0; ks < C::KS; ++ks) mma(acc, kc[tb][ks], wf[mb][ks]);
#pragma unroll
        for (int j = 0; j < 4; ++j) uu[8 * mb + 4 * tb + j] = acc[j] + bcol[mb];
      }
    int sg[8 * MB];
    pwl_search(tab, tsteps, uu, sg);
    Frag<T> af[MB][L];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const bool pok = 16 * mb + r < M;
#pragma unroll
      for (int e = 0; e < 8; ++e) {  // slot e = 4 tb + j
        const bool ok = pok && (t0 + 16 * (e / 4) + 4 * g + (e % 4) < t_end);
        float y[L];
        pwl_channels<L>(tab, sg[8 * mb + e], tfloor, uu[8 * mb + e], y);
#pragma unroll
        for (int l = 0; l < L; ++l) af[mb][l].set(e, ok ? y[l] : 0.0f);
      }
    }
    // S += phi(K)^T V, z += phi(K)^T 1
#pragma unroll
    for (int cb = 0; cb < C::CB; ++cb) {
      Frag<T> bv;
      load4(bv, 0, &vt[wave][16 * cb + r][4 * g]);
      load4(bv, 4, &vt[wave][16 * cb + r][16 + 4 * g]);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int l = 0; l < L; ++l) mma(accS[mb][l][cb], af[mb][l], bv);
    }
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int l = 0; l < L; ++l) mma(accZ[mb][l], af[mb][l], ones);
    __syncthreads();
  }

  // sum the four waves in a fixed order
  for (int w = 0; w < 4; ++w) {
    if (wave == w) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int l = 0; l < L; ++l)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int row = (mb * L + l) * 16 + 4 * g + j;
#pragma unroll
            for (int cb = 0; cb < C::CB; ++cb) {
              float& d = red[row][16 * cb + r];
              d = (w == 0) ? accS[mb][l][cb][j] : d + accS[mb][l][cb][j];
            }
            if (r == 0) {
              float& d = red[row][DH];
              d = (w == 0) ? accZ[mb][l][j] : d + accZ[mb][l][j];
            }
          }
    }
    __syncthreads();
  }
  float* part = a.partial + ((size_t)head * a.splits + split) * C::DP * (DH + 1);
  const float* src = &red[0][0];
  for (int i = threadIdx.x; i < C::DP * (DH + 1); i += blockDim.x) part[i] = src[i];
}

// ---------------------------------------------------------------------------
// reduce pass: partials -> readout fragments
// ---------------------------------------------------------------------------
template <typename T, int DH, int L, int MB>
__global__ __launch_bounds__(256) void nc_reduce_kernel(NoncausalArgs a) {
  using C = NcCfg<T, DH, L, MB>;
  // blockIdx.y: a slice of the head's fragment elements; every element sums its own
  // partials in range order (deterministic), so the slices need no exchange
  const int head = blockIdx.x;
  const float* part = a.partial + (size_t)head * a.splits * C::DP * (DH + 1);
  T* fr = reinterpret_cast<T*>(a.frags) + (size_t)head * C::FRAG_ELEMS;
  // fragment (cb, kappa), lane (g, r), slot e; cb == CB holds z
  for (size_t idx = (size_t)blockIdx.y * blockDim.x + threadIdx.x; idx < C::FRAG_ELEMS;
       idx += (size_t)gridDim.y * blockDim.x) {
    const int e = (int)(idx % 8);
    const int lane = (int)((idx / 8) % kWave);
    const int kappa = (int)((idx / (8 * kWave)) % C::NF);
    const int cb = (int)(idx / (8 * kWave * C::NF));
    const int g = lane / 16, r = lane % 16;
    const int p = 8 * kappa + e;
    float v = 0.0f;
    if (p < 4 * MB * L) {
      const int mbj = p / L, l = p % L;
      const int mb = mbj / 4, j = mbj % 4;
      const int row = (mb * L + l) * 16 + 4 * g + j;
      const int src = row * (DH + 1) + (cb < C::CB ? 16 * cb + r : DH);
      for (int sp = 0; sp < a.splits; ++sp) v += part[(size_t)sp * C::DP * (DH + 1) + src];
    }
    fr[idx] = (T)v;
  }
}

// ---------------------------------------------------------------------------
// state export: the partials summed in range order into S [D][d] and z [D]
// (feature i*L + l, fp32, the coefficient rows' power-of-two scale removed), or
// added to them
// ---------------------------------------------------------------------------
template <typename T, int DH, int L, int MB>
__global__ __launch_bounds__(256) void nc_state_export_kernel(NoncausalArgs a) {
  using C = NcCfg<T, DH, L, MB>;
  const int head = blockIdx.x;
  const int hset = a.phi.per_head ? head % a.H : 0;
  const PwlHeader hd = *reinterpret_cast<const PwlHeader*>(a.phi.tables + (size_t)hset * kTableBytes + kTabHeader);
  // the state pass evaluates bf16 data with fp16 rows that hold 2^scale_exp times the values
  const float unscale = sizeof(T) == 2 ? ldexpf(1.0f, -hd.scale_exp) : 1.0f;
  const int M = a.phi.M;
  const float* part = a.partial + (size_t)head * a.splits * C::DP * (DH + 1);
  float* S = a.state_S + (size_t)head * M * L * DH;
  float* z = a.state_z + (size_t)head * M * L;
  for (int i = blockIdx.y * blockDim.x + threadIdx.x; i < C::DP * (DH + 1); i += gridDim.y * blockDim.x) {
    const int row = i / (DH + 1), col = i % (DH + 1);
    // partial row (mb, l, i16) holds projection 16 mb + i16, channel l
    const int mb = row / (16 * L), l = (row / 16) % L, p = 16 * mb + row % 16;
    if (p >= M) continue;
    float v = 0.0f;
    for (int sp = 0; sp < a.splits; ++sp) v += part[(size_t)sp * C::DP * (DH + 1) + i];
    v *= unscale;
    const int f = p * L + l;
    float* dst = col < DH ? &S[(size_t)f * DH + col] : &z[f];
    *dst = a.accumulate ? *dst + v : v;
  }
}

// ---------------------------------------------------------------------------
// readout pass
// ---------------------------------------------------------------------------
template <typename T, int DH, int L, int MB>
__global__ __launch_bounds__(256, 1) void nc_readout_kernel(NoncausalArgs a) {
  using C = NcCfg<T, DH, L, MB>;
  __shared__ typename PwlTab<T, L, C::NSEG>::type tab;
  const int head = blockIdx.x / a.tiles;
  const int tile = blockIdx.x - head * a.tiles;
  const int hset = a.phi.per_head ? head % a.H : 0;
  pwl_load(tab, a.phi.tables + (size_t)hset * kTableBytes);

  const int wave = wave_id(), lane = threadIdx.x % kWave;
  const int g = lane / 16, r = lane % 16;
  const int M = a.phi.M;
  const size_t hoff = (size_t)head * a.n * DH;
  const T* Q = reinterpret_cast<const T*>(a.Q) + hoff;
  T* out = reinterpret_cast<T*>(a.out) + hoff;
  const T* W = reinterpret_cast<const T*>(a.phi.W) + (size_t)hset * M * DH;
  const float* bias = a.phi.b + (size_t)hset * M;
  const T* fr = reinterpret_cast<const T*>(a.frags) + (size_t)head * C::FRAG_ELEMS;

  Frag<T> sf[C::CB][C::NF], zf[C::NF];
#pragma unroll
  for (int cb = 0; cb < C::CB; ++cb)
#pragma unroll
    for (int k = 0; k < C::NF; ++k) load8(sf[cb][k], fr + ((size_t)(cb * C::NF + k) * kWave + lane) * 8);
#pragma unroll
  for (int k = 0; k < C::NF; ++k) load8(zf[k], fr + ((size_t)(C::CB * C::NF + k) * kWave + lane) * 8);

  // A operand of u^T = W Q^T: row r of block mb is projection 16mb + r.
  Frag<T> wf[MB][C::KS];
  float brow[MB][4];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int p = 16 * mb + r;
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      if (p < M) load8(wf[mb][ks], W + (size_t)p * DH + 32 * ks + 8 * g);
      else wf[mb][ks].zero();
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = 16 * mb + 4 * g + j;
      brow[mb][j] = i < M ? bias[i] : 0.0f;
    }
  }
  __syncthreads();
  const int tsteps = __builtin_amdgcn_readfirstlane(tab.steps);
  const float tfloor = tab.floor;

  const int nblk = a.tile_tokens / 16;
  for (int blk = wave; blk < nblk; blk += 4) {
    const int t = tile * a.tile_tokens + blk * 16 + r;
    const bool ok = t < a.n;
    Frag<T> qf[C::KS];
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      if (ok) load8(qf[ks], Q + (size_t)t * DH + 32 * ks + 8 * g);
      else qf[ks].zero();
    }
    Frag<T> pq[C::NF];
#pragma unroll
    for (int k = 0; k < C::NF; ++k) pq[k].zero();
    float uu[4 * MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      f32x4 acc = zero4();
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) mma(acc, wf[mb][ks], qf[ks]);
#pragma unroll
      for (int j = 0; j < 4; ++j) uu[4 * mb + j] = acc[j] + brow[mb][j];
    }
    int sg[4 * MB];
    pwl_search(tab, tsteps, uu, sg);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bool pok = 16 * mb + 4 * g + j < M;
        float y[L];
        pwl_channels<L>(tab, sg[4 * mb + j], tfloor, uu[4 * mb + j], y);
#pragma unroll
        for (int l = 0; l < L; ++l) {
          const int p = (mb * 4 + j) * L + l;
          pq[p / 8].set(p % 8, pok ? y[l] : 0.0f);
        }
      }
    }
    f32x4 num[C::CB], den = zero4();
#pragma unroll
    for (int cb = 0; cb < C::CB; ++cb) num[cb] = zero4();
#pragma unroll
    for (int k = 0; k < C::NF; ++k) {
#pragma unroll
      for (int cb = 0; cb < C::CB; ++cb) mma(num[cb], sf[cb][k], pq[k]);
      mma(den, zf[k], pq[k]);
    }
    if (ok) {
      const float rinv = 1.0f / (den[0] + ldexpf(a.eps, 2 * tab.scale_exp));
      T* o = out + (size_t)t * DH + 4 * g;
#pragma unroll
      for (int cb = 0; cb < C::CB; ++cb)
        store4(o + 16 * cb, num[cb][0] * rinv, num[cb][1] * rinv, num[cb][2] * rinv, num[cb][3] * rinv);
    }
  }
}


// ---------------------------------------------------------------------------
// fused pass: one workgroup of kNcWaves waves per head (used when there are enough heads
// to fill the device).  The state phase accumulates each wave's share of S and z
// in registers (phi(K) fragments never leave registers; V is read transposed from
// a wave-private row-major LDS tile); the waves are summed in LDS in a fixed order
// and converted to readout fragments; the readout phase then streams the head's
// queries with S and z held in registers.  S never reaches HBM.
// ---------------------------------------------------------------------------
constexpr int kNcWaves = 4;  // one wave per SIMD: the whole register file per wave

template <typename T, int DH, int L, int MB>
struct NcFusedLds {
  using C = NcCfg<T, DH, L, MB>;
  static constexpr int VR = DH + C::VE;   // padded V-tile row (elements)
  static constexpr int NTILE = MB * L * C::CB + MB;  // accumulator tiles of S, then of z
  // one channel per projection (a lookup per feature, so the lookups set the pace): the
  // fp16-row table with every bucket's first comparison key, one dependent LDS read
  // fewer per lookup (455 -> 393 us on the long encoder problem's one-channel map).
  // With eight channels per lookup the 12 KB more that every workgroup copies cost more
  // than the read saves (text encoder 58.1 -> 60.2 us).
  typename std::conditional<sizeof(T) == 2 && L == 1, PwlLds16F<L, C::NSEG>,
                            typename PwlTab<T, L, C::NSEG>::type>::type tab;
  union {
    T vt[kNcWaves][32][VR];             // per-wave V tile of the current 32-token step
    float4 red[NTILE][kWave];           // cross-wave sum of the accumulator tiles, lane-major
  } u;
};

template <typename T, int DH, int L, int MB>
__global__ __launch_bounds__(64 * kNcWaves, 1) void nc_fused_kernel(NoncausalArgs a) {
  using C = NcCfg<T, DH, L, MB>;
  using LDS = NcFusedLds<T, DH, L, MB>;
  __shared__ LDS sm;

  const int head = blockIdx.x;
  const int hset = a.phi.per_head ? head % a.H : 0;
  pwl_load(sm.tab, a.phi.tables + (size_t)hset * kTableBytes);

  const int wave = wave_id(), lane = threadIdx.x % kWave;
  const int g = lane / 16, r = lane % 16;
  const int M = a.phi.M;
  const int n = a.n;
  const size_t hoff = (size_t)head * n * DH;
  const T* Q = reinterpret_cast<const T*>(a.Q) + hoff;
  const T* K = reinterpret_cast<const T*>(a.K) + hoff;
  const T* V = reinterpret_cast<const T*>(a.V) + hoff;
  T* out = reinterpret_cast<T*>(a.out) + hoff;
  const T* W = reinterpret_cast<const T*>(a.phi.W) + (size_t)hset * M * DH;
  const float* bias = a.phi.b + (size_t)hset * M;

  // W fragments: lane index r of block mb is projection 16mb + r (B of u = K W^T,
  // A of u^T = W Q^T)
  Frag<T> wf[MB][C::KS];
  float bcol[MB], brow[MB][4];
  bool pcol[MB], prow[MB][4];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int p = 16 * mb + r;
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      if (p < M) load8(wf[mb][ks], W + (size_t)p * DH + 32 * ks + 8 * g);
      else wf[mb][ks].zero();
    }
    pcol[mb] = p < M;
    bcol[mb] = p < M ? bias[p] : 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = 16 * mb + 4 * g + j;
      prow[mb][j] = i < M;
      brow[mb][j] = i < M ? bias[i] : 0.0f;
    }
  }
  Frag<T> ones;
  ones.fill(1.0f);

  // z of channel l is accumulated in column l of accZ[mb] (B = one-hot column l)
  static_assert(L <= 16, "one accumulator column per channel");
  f32x4 accS[MB][L][C::CB];
  f32x4 accZ[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    accZ[mb] = zero4();
#pragma unroll
    for (int l = 0; l < L; ++l)
#pragma unroll
      for (int cb = 0; cb < C::CB; ++cb) accS[mb][l][cb] = zero4();
  }

  // ---- state phase: wave w takes 32-token steps w, w + kNcWaves, ... ----
  constexpr int VCH = 32 * DH / C::VE / kWave;  // V 16-byte chunks per lane per step
  Frag<T> kn[2][C::KS], kq[2][C::KS];  // this step's K rows, the next step's
  i32x4 vn[VCH];
  // rows of a 32-token step through range-checked buffers (rows past n read as 0)
  auto fetch_k = [&](Frag<T> (&kf)[2][C::KS], int step) {
    const auto rs = rows_rsrc(K, 32 * step, 32, n, DH, (int)sizeof(T));
#pragma unroll
    for (int tb = 0; tb < 2; ++tb)
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks)
        buf_load8(kf[tb][ks], rs, (int)(((16 * tb + r) * DH + 32 * ks + 8 * g) * sizeof(T)));
  };
  auto fetch_v = [&](int step) {
    const auto rs = rows_rsrc(V, 32 * step, 32, n, DH, (int)sizeof(T));
#pragma unroll
    for (int q = 0; q < VCH; ++q) {
      const int c = lane + kWave * q;
      const int tt = c / (DH / C::VE), cg = c % (DH / C::VE);
      vn[q] = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                            rs, (int)((tt * DH + cg * C::VE) * sizeof(T)), 0, 0));
    }
  };
  __syncthreads();
  const int tsteps = __builtin_amdgcn_readfirstlane(sm.tab.steps);
  const int zseg = sm.tab.zero_seg;
  const float tfloor = sm.tab.floor;
  T* vt = &sm.u.vt[wave][0][0];

  const int nsteps = (n + 31) / 32;
  // loads are issued on every path (past the last step as empty buffers), so that the
  // waits for them count the same loads on every path; a step's rows are fetched one
  // whole step ahead
  fetch_k(kn, wave);
  fetch_v(wave);
  for (int step = wave; step < nsteps; step += kNcWaves) {
    const int t0 = 32 * step;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
#pragma unroll
    for (int q = 0; q < VCH; ++q) {
      const int c = lane + kWave * q;
      const int tt = c / (DH / C::VE), cg = c % (DH / C::VE);
      *reinterpret_cast<i32x4*>(vt + tt * LDS::VR + cg * C::VE) = vn[q];
    }
    fetch_v(step + kNcWaves);
    fetch_k(kq, step + kNcWaves);

    float uu[8 * MB];  // [mb][tb][j]
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        f32x4 acc = zero4();
#pragma unroll
        for (int ks = 0; ks < C::KS; ++ks) mma(acc, kn[tb][ks], wf[mb][ks]);
#pragma unroll
        for (int j = 0; j < 4; ++j) uu[8 * mb + 4 * tb + j] = acc[j] + bcol[mb];
      }
    int sg[8 * MB];
    pwl_search(sm.tab, tsteps, uu, sg);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int e = 0; e < 8; ++e)  // slot e = 4 tb + j holds token t0 + 16 tb + 4 g + j
        if (!pcol[mb] || t0 + 16 * (e / 4) + 4 * g + (e % 4) >= n) sg[8 * mb + e] = zseg;
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    Frag<T> bv[C::CB];
#pragma unroll
    for (int cb = 0; cb < C::CB; ++cb) {
      load_tr4(bv[cb], 0, vt, LDS::VR, 4 * g, 16 * cb, lane);
      load_tr4(bv[cb], 4, vt, LDS::VR, 16 + 4 * g, 16 * cb, lane);
    }
    // each value's argument on its segment, taken once for the L / 2 channel pairs (after
    // the V tile's fence, so that the anchors, the coefficient rows and the V fragments
    // are read in one round trip)
    float xx[8 * MB];
#pragma unroll
    for (int v = 0; v < 8 * MB; ++v) xx[v] = pwl_local(sm.tab, sg[v], uu[v]);
    // channel pairs: evaluate the 8 token slots, multiply, drop
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      if constexpr (L % 2 == 0) {
#pragma unroll
        for (int q = 0; q < L / 2; ++q) {
          Frag<T> a0, a1;
#pragma unroll
          for (int e = 0; e < 8; e += 2) {
            float y00, y01, y10, y11;
            pwl_pair_local<L>(sm.tab, sg[8 * mb + e], q, tfloor, xx[8 * mb + e], y00, y01);
            pwl_pair_local<L>(sm.tab, sg[8 * mb + e + 1], q, tfloor, xx[8 * mb + e + 1], y10, y11);
            a0.set2(e, y00, y10);
            a1.set2(e, y01, y11);
          }
#pragma unroll
          for (int cb = 0; cb < C::CB; ++cb) {
            mma(accS[mb][2 * q][cb], a0, bv[cb]);
            mma(accS[mb][2 * q + 1][cb], a1, bv[cb]);
          }
          Frag<T> oh0, oh1;
          oh0.fill(r == 2 * q ? 1.0f : 0.0f);
          oh1.fill(r == 2 * q + 1 ? 1.0f : 0.0f);
          mma(accZ[mb], a0, oh0);
          mma(accZ[mb], a1, oh1);
        }
      } else {
#pragma unroll
        for (int l = 0; l < L; ++l) {
          Frag<T> a0;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            float y[L];
            pwl_channels<L>(sm.tab, sg[8 * mb + e], tfloor, uu[8 * mb + e], y);
            a0.set(e, y[l]);
          }
#pragma unroll
          for (int cb = 0; cb < C::CB; ++cb) mma(accS[mb][l][cb], a0, bv[cb]);
          Frag<T> oh;
          oh.fill(r == l ? 1.0f : 0.0f);
          mma(accZ[mb], a0, oh);
        }
      }
    }
#pragma unroll
    for (int tb = 0; tb < 2; ++tb)
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) kn[tb][ks] = kq[tb][ks];
  }

  // ---- readout rows: wave w takes 16-token blocks w, w + kNcWaves, ... ----
  const int nblk = (n + 15) / 16;
  // NB query blocks are mapped together, so that their table lookups overlap (one wave
  // per SIMD has no other wave to hide their latency); blocks past the end read zero
  // rows and store nothing.  The next group's rows are fetched while one is mapped.
  // Loads and stores share one counter and their completions are not ordered, so a
  // wait for a load also waits for every store issued before it: the group's outputs
  // are kept until its end and stored after an explicit wait for the next group's
  // rows, so that no wait has to cover stores issued just before it.
  constexpr int NB = 2;
  Frag<T> qf[NB][C::KS];
  auto fetch_q = [&](Frag<T> (&qf)[C::KS], int b) {
    const auto rs = rows_rsrc(Q, 16 * b, 16, n, DH, (int)sizeof(T));
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) buf_load8(qf[ks], rs, (int)((r * DH + 32 * ks + 8 * g) * sizeof(T)));
  };
#pragma unroll
  for (int i = 0; i < NB; ++i) fetch_q(qf[i], wave + kNcWaves * i);
  // ---- sum the waves' accumulator tiles in a fixed order (deterministic), lane by
  // lane: every tile is one 16-byte read-modify-write per lane ----
  __syncthreads();  // every wave is done with its V tile (red aliases it)
  for (int w = 0; w < kNcWaves; ++w) {
    if (wave == w) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
        for (int l = 0; l < L; ++l)
#pragma unroll
          for (int cb = 0; cb < C::CB; ++cb) {
            float4& d = sm.u.red[(mb * L + l) * C::CB + cb][lane];
            const f32x4 v = accS[mb][l][cb];
            d = (w == 0) ? make_float4(v[0], v[1], v[2], v[3])
                         : make_float4(d.x + v[0], d.y + v[1], d.z + v[2], d.w + v[3]);
          }
        float4& d = sm.u.red[MB * L * C::CB + mb][lane];
        const f32x4 v = accZ[mb];
        d = (w == 0) ? make_float4(v[0], v[1], v[2], v[3])
                     : make_float4(d.x + v[0], d.y + v[1], d.z + v[2], d.w + v[3]);
      }
    }
    __syncthreads();
  }
  // Readout fragments.  Tile (mb, l, cb), lane (g, r), element j holds S[feature
  // (mb, projection 16 mb + 4 g + j, channel l)][column 16 cb + r]; readout fragment
  // kappa, slot e of the same lane is list position p = 8 kappa + e = (4 mb + j) L + l
  // of that lane's group, column 16 cb + r: the same value, no lane exchange.  z
  // (tile column l = channel l) is gathered across lanes: every row of its fragment
  // is z.
  Frag<T> sf[C::CB][C::NF], zf[C::NF];
#pragma unroll
  for (int cb = 0; cb < C::CB; ++cb)
#pragma unroll
    for (int k = 0; k < C::NF; ++k) sf[cb][k].zero();
#pragma unroll
  for (int k = 0; k < C::NF; ++k) zf[k].zero();
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int l = 0; l < L; ++l)
#pragma unroll
      for (int cb = 0; cb < C::CB; ++cb) {
        const float4 v = sm.u.red[(mb * L + l) * C::CB + cb][lane];
        const float vj[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int p = (4 * mb + j) * L + l;
          sf[cb][p / 8].set(p % 8, vj[j]);
        }
      }
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int l = 0; l < L; ++l) {
      const float4 v = sm.u.red[MB * L * C::CB + mb][16 * g + l];  // lane (g, l): channel l
      const float vj[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int p = (4 * mb + j) * L + l;
        zf[p / 8].set(p % 8, vj[j]);
      }
    }

  // ---- readout phase: wave w takes 16-token blocks w, w + kNcWaves, ... ----
  // (the first group's rows were fetched before the reduction; every load issued so
  // far is complete from here on, so the loop's waits see only its own accesses)
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  for (int b0 = wave; b0 < nblk; b0 += kNcWaves * NB) {
    float uu[NB * 4 * MB];  // [block][mb][j]
#pragma unroll
    for (int i = 0; i < NB; ++i)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        f32x4 acc = zero4();
#pragma unroll
        for (int ks = 0; ks < C::KS; ++ks) mma(acc, wf[mb][ks], qf[i][ks]);
#pragma unroll
        for (int j = 0; j < 4; ++j) uu[(i * MB + mb) * 4 + j] = acc[j] + brow[mb][j];
      }
#pragma unroll
    for (int i = 0; i < NB; ++i) fetch_q(qf[i], b0 + kNcWaves * (NB + i));  // rows projected: next group
    int sg[NB * 4 * MB];
    pwl_search(sm.tab, tsteps, uu, sg);
#pragma unroll
    for (int i = 0; i < NB; ++i)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (!prow[mb][j]) sg[(i * MB + mb) * 4 + j] = zseg;
    f32x4 num[NB][C::CB], den[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      Frag<T> pq[C::NF];
#pragma unroll
      for (int k = 0; k < C::NF; ++k) pq[k].zero();
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int v = (i * MB + mb) * 4 + j;
          float y[L];
          pwl_channels<L>(sm.tab, sg[v], tfloor, uu[v], y);
#pragma unroll
          for (int l = 0; l < L; ++l) {
            const int p = (mb * 4 + j) * L + l;
            if constexpr (L % 2 == 0) {
              if (l % 2 == 0) pq[p / 8].set2(p % 8, y[l], y[l + 1]);
            } else {
              pq[p / 8].set(p % 8, y[l]);
            }
          }
        }
      den[i] = zero4();
#pragma unroll
      for (int cb = 0; cb < C::CB; ++cb) num[i][cb] = zero4();
#pragma unroll
      for (int k = 0; k < C::NF; ++k) {
#pragma unroll
        for (int cb = 0; cb < C::CB; ++cb) mma(num[i][cb], sf[cb][k], pq[k]);
        mma(den[i], zf[k], pq[k]);
      }
    }
    // the next group's rows and the previous group's stores, before this group's stores
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      // rows past n are dropped by the range-checked buffer
      const auto ro = rows_rsrc(out, 16 * (b0 + kNcWaves * i), 16, n, DH, (int)sizeof(T));
      const float rinv = __builtin_amdgcn_rcpf(den[i][0] + ldexpf(a.eps, 2 * sm.tab.scale_exp));
#pragma unroll
      for (int cb = 0; cb < C::CB; ++cb)
        buf_store4<T>(ro, (int)((r * DH + 16 * cb + 4 * g) * sizeof(T)), num[i][cb][0] * rinv,
                      num[i][cb][1] * rinv, num[i][cb][2] * rinv, num[i][cb][3] * rinv);
    }
  }
}

// ---------------------------------------------------------------------------
// dispatch
// ---------------------------------------------------------------------------
template <typename T, int DH, int L, int MB>
static hipError_t nc_run(const NoncausalArgs& a, hipStream_t s) {
  if constexpr (fused_acc_regs(DH, L, 16 * MB) <= kFusedMaxAccRegs) {
    if (a.fused) {
      hipLaunchKernelGGL((nc_fused_kernel<T, DH, L, MB>), dim3(a.heads), dim3(64 * kNcWaves), 0, s, a);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((nc_state_kernel<T, DH, L, MB>), dim3(a.heads * a.splits), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  {
    using C = NcCfg<T, DH, L, MB>;
    constexpr int kSlices = (int)((C::FRAG_ELEMS + 255) / 256);
    hipLaunchKernelGGL((nc_reduce_kernel<T, DH, L, MB>), dim3(a.heads, kSlices), dim3(256), 0, s, a);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((nc_readout_kernel<T, DH, L, MB>), dim3(a.heads * a.tiles), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename T, int DH, int L, int MB>
static hipError_t state_run(const NoncausalArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((nc_state_kernel<T, DH, L, MB>), dim3(a.heads * a.splits), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((nc_state_export_kernel<T, DH, L, MB>), dim3(a.heads, 8), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename T, int DH, int L, int MB>
static void nc_plan(NoncausalPlan* p) {
  using C = NcCfg<T, DH, L, MB>;
  p->DP = C::DP;
  p->NF = C::NF;
  p->frag_elems = C::FRAG_ELEMS;
}

// (dtype, d, L, projection blocks) combinations that are built.
#define LUNA_NC_CASES(X)   \
  X(float, 32, 8, 1)       \
  X(float, 32, 2, 1)       \
  X(float, 64, 8, 1)       \
  X(__bf16, 32, 8, 1)      \
  X(__bf16, 64, 8, 1)      \
  X(__bf16, 64, 8, 2)      \
  X(__bf16, 64, 4, 1)      \
  X(__bf16, 64, 1, 4)      \
  X(__bf16, 64, 1, 8)      \
  X(__bf16, 128, 8, 1)

template <typename T>
static constexpr Dt dt_of() { return sizeof(T) == 2 ? Dt::BF16 : Dt::F32; }

bool noncausal_supported(Dt dt, int d, int L, int M, NoncausalPlan* plan) {
  const int MB = (M + 15) / 16;
#define X(T_, D_, L_, MB_)                                              \
  if (dt == dt_of<T_>() && d == D_ && L == L_ && MB == MB_) {           \
    if (plan) nc_plan<T_, D_, L_, MB_>(plan);                           \
    return true;                                                        \
  }
  LUNA_NC_CASES(X)
#undef X
  return false;
}

hipError_t launch_state(Dt dt, int d, int L, int M, const NoncausalArgs& a, hipStream_t s) {
  const int MB = (M + 15) / 16;
#define X(T_, D_, L_, MB_) \
  if (dt == dt_of<T_>() && d == D_ && L == L_ && MB == MB_) return state_run<T_, D_, L_, MB_>(a, s);
  LUNA_NC_CASES(X)
#undef X
  return hipErrorInvalidValue;
}

hipError_t launch_noncausal(Dt dt, int d, int L, int M, const NoncausalArgs& a, hipStream_t s) {
  const int MB = (M + 15) / 16;
#define X(T_, D_, L_, MB_) \
  if (dt == dt_of<T_>() && d == D_ && L == L_ && MB == MB_) return nc_run<T_, D_, L_, MB_>(a, s);
  LUNA_NC_CASES(X)
#undef X
  return hipErrorInvalidValue;
}

}  // namespace luna
