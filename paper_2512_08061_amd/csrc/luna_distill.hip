// luna_distill.hip -- the attention-distillation loss of the conversion recipe's first
// stage (Implementation Details appendix: the feature map alone is trained so that
// LUNA's attention distribution matches the teacher's softmax attention, eq. (1) of
// Section 2), and its gradient with respect to the features.
//
// Per query row t, with the keys s that t sees (all, or s <= t when causal; n_t of them):
//   teacher  A_ts = softmax_s(q_t . k_s / sqrt(d))
//   student  Ahat_ts = (P_ts + eps / n_t) / (den_t + eps),  P = phi(Q) phi(K)^T,
//            den_t = sum_s P_ts  (LUNA's weights of eq. (9), smoothed into an exact
//            distribution)
//   loss     CE_t = -sum_s A_ts log Ahat_ts = -sum_s A_ts log(P_ts + eps / n_t) + log(den_t + eps)
// and for the mean over the N rows of the call
//   G_ts = (1/N) (1 / (den_t + eps) - A_ts / (P_ts + eps / n_t)),
//   dphi(q_t) = sum_s G_ts phi(k_s),  dphi(k_s) = sum_t G_ts phi(q_t).
//
// Flash-style: nothing of size n x n is stored.  distill_q_kernel takes 64 queries per
// workgroup (16 per wave) and walks the key tiles once, with the softmax maximum kept
// online (base 2) and every sum taken against it rescaled as it grows: the softmax sum,
// den, the loss and dphi(Q).  distill_k_kernel takes
// 64 keys per workgroup and walks the query tiles once for dphi(K), from the per-row
// statistics the first kernel stored.  Per tile, S^T = K Q^T and P^T = phi(K) phi(Q)^T
// run on the matrix cores with the wave's queries as the B operand held in registers,
// so that each lane holds 16 keys of one query; the gradient products take G straight
// from those registers as the A operand, its 32 keys in the order lane group g holds
// them ({4g..4g+3} and {16+4g..16+4g+3} of each 32), with the matching rows of the
// staged feature tile read transposed (the gfx950 transpose read for bf16).  bf16 calls
// use bf16 matrix-core products with fp32 accumulation and split G into two bf16 parts;
// fp32 calls use the fp32 matrix cores.
#include <math.h>

#include "luna_device.hpp"
#include "luna_kernels.hpp"

namespace luna {

namespace {

constexpr float kLog2e = 1.44269504088896341f;
constexpr float kLn2 = 0.693147180559945309f;

// The hardware's base-2 exponential, base-2 logarithm and reciprocal (about 1 ulp on
// normal fp32 values).  Exponentials below 2^-126 come out as 0 (a softmax weight that
// small against the row's maximum changes no sum) and a logarithm or reciprocal of a
// value below 2^-126 is taken as of 0: P + eps / n_t only gets there when eps is below
// n 2^-126, i.e. in effect eps = 0, where such a key's loss is infinite either way.
__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float lg2(float x) { return __builtin_amdgcn_logf(x); }
__device__ __forceinline__ float rcp(float x) { return __builtin_amdgcn_rcpf(x); }

// Workgroups are dealt to the eight XCDs in turn (workgroup b to XCD b mod 8), each
// XCD with its own L2.  Workgroup b's work item is renumbered so that every XCD takes
// one contiguous run of items, first to last in dispatch order: the 64-row tiles of a
// head, which all read the same tiles of the other side, then share one L2.  (A
// bijection of [0, items) for any count.)
__device__ __forceinline__ int64_t xcd_item(int64_t b, int64_t items) {
  constexpr int64_t kXcds = 8;
  const int64_t per = items / kXcds, rem = items % kXcds, x = b % kXcds, i = b / kXcds;
  return x < rem ? x * (per + 1) + i : rem * (per + 1) + (x - rem) * per + i;
}

// Compile-time flag of a tile in which every key is visible to every query.
template <bool B>
struct Whole {
  static constexpr bool value = B;
};

template <typename T, int DH, int DF>
struct DistShape {
  static constexpr int PAD = 16 / (int)sizeof(T);  // one 16-byte chunk per row
  static constexpr int LDH = DH + PAD, LDF = DF + PAD;
  static constexpr int KD = DH / 32, KF = DF / 32, NFO = DF / 16;
};

// Rows r0 .. r0 + 63 of two row-major arrays, [n][W1] and [n][W2] of T, for LDS tiles
// with row strides LD1 and LD2 (rows at or past n as zeros), 16 bytes per thread and
// step of the 256 threads.  load() issues every global read into registers and store()
// writes them to the tiles, so a tile costs one memory round trip, and reads issued
// before the barrier that frees the tiles are in flight while the workgroup waits.
template <typename T, int W1, int LD1, int W2, int LD2>
struct TileRows {
  static constexpr int CH1 = W1 * (int)sizeof(T) / 16, CH2 = W2 * (int)sizeof(T) / 16;
  static constexpr int IT1 = 64 * CH1 / 256, IT2 = 64 * CH2 / 256;
  static_assert(IT1 * 256 == 64 * CH1 && IT2 * 256 == 64 * CH2, "whole 256-thread steps");
  uint4 v1[IT1], v2[IT2];
  __device__ __forceinline__ void load(const T* src1, const T* src2, int64_t r0, int64_t n, int tid) {
#pragma unroll
    for (int it = 0; it < IT1; ++it) {
      const int i = tid + 256 * it, row = i / CH1, c = i % CH1;
      v1[it] = uint4{0u, 0u, 0u, 0u};
      if (r0 + row < n) v1[it] = *reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(src1 + (r0 + row) * W1) + 16 * c);
    }
#pragma unroll
    for (int it = 0; it < IT2; ++it) {
      const int i = tid + 256 * it, row = i / CH2, c = i % CH2;
      v2[it] = uint4{0u, 0u, 0u, 0u};
      if (r0 + row < n) v2[it] = *reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(src2 + (r0 + row) * W2) + 16 * c);
    }
  }
  __device__ __forceinline__ void store(T* tile1, T* tile2, int tid) const {
#pragma unroll
    for (int it = 0; it < IT1; ++it) {
      const int i = tid + 256 * it, row = i / CH1, c = i % CH1;
      *reinterpret_cast<uint4*>(reinterpret_cast<char*>(tile1 + row * LD1) + 16 * c) = v1[it];
    }
#pragma unroll
    for (int it = 0; it < IT2; ++it) {
      const int i = tid + 256 * it, row = i / CH2, c = i % CH2;
      *reinterpret_cast<uint4*>(reinterpret_cast<char*>(tile2 + row * LD2) + 16 * c) = v2[it];
    }
  }
};

// The gradient values of one 32-wide k block as an A fragment (slots 0..3 from the
// first 16-block's four values, 4..7 from the second's); bf16 splits each value into
// a high and a low bf16 part.
template <typename T>
struct GFrag {
  Frag<T> hi, lo;
  __device__ __forceinline__ void set(const float (&g0)[4], const float (&g1)[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      hi.set(j, g0[j]);
      hi.set(4 + j, g1[j]);
      if constexpr (sizeof(T) == 2) {
        lo.set(j, g0[j] - hi.get(j));
        lo.set(4 + j, g1[j] - hi.get(4 + j));
      }
    }
  }
  __device__ __forceinline__ void apply(f32x4& acc, const Frag<T>& b) const {
    mma(acc, hi, b);
    if constexpr (sizeof(T) == 2) mma(acc, lo, b);
  }
};

// Waves per SIMD: the bf16 loss alone keeps 4 (3 at D = 256, where the LDS tiles allow
// no more); fp32 tiles and the gradients' accumulators leave room for 2.
template <typename T, int DH, int DF, bool GRAD>
__global__ __launch_bounds__(256, GRAD || sizeof(T) == 4 ? 2 : (DF <= 128 ? 4 : 3)) void distill_q_kernel(DistillArgs a) {
  using S = DistShape<T, DH, DF>;
  __shared__ __align__(16) T sk[64 * S::LDH];
  __shared__ __align__(16) T sf[64 * S::LDF];
  const int tid = threadIdx.x, wave = wave_id(), lane = tid % kWave;
  const int g = lane / 16, r = lane % 16;
  const int64_t n = a.n;
  const int ntiles = (int)((n + 63) / 64);
  const int64_t item = xcd_item(blockIdx.x, gridDim.x);
  const int64_t head = item / ntiles;
  // causal: the last query tiles (the most key tiles) are dispatched first
  const int qt = a.causal ? ntiles - 1 - (int)(item - head * ntiles) : (int)(item - head * ntiles);
  const int64_t tq = (int64_t)qt * 64 + wave * 16 + r;  // this lane's query
  const bool q_ok = tq < n;
  const T* Kh = reinterpret_cast<const T*>(a.K) + head * n * DH;
  const T* Fk = reinterpret_cast<const T*>(a.phik) + head * n * DF;
  Frag<T> qf[S::KD], ff[S::KF];
  {
    const T* q = reinterpret_cast<const T*>(a.Q) + (head * n + (q_ok ? tq : 0)) * DH;
    const T* f = reinterpret_cast<const T*>(a.phiq) + (head * n + (q_ok ? tq : 0)) * DF;
#pragma unroll
    for (int kb = 0; kb < S::KD; ++kb) {
      if (q_ok) load8(qf[kb], q + 32 * kb + 8 * g);
      else qf[kb].zero();
    }
#pragma unroll
    for (int kb = 0; kb < S::KF; ++kb) {
      if (q_ok) load8(ff[kb], f + 32 * kb + 8 * g);
      else ff[kb].zero();
    }
  }
  const float c2 = a.scale * kLog2e;  // logits in base 2
  const int last = a.causal ? qt : ntiles - 1;
  const float eps_nt = a.eps / (float)(a.causal ? tq + 1 : n);

  // S^T and P^T of key tile kt: st[c][j], pt[c][j] for key 64 kt + 16 c + 4 g + j
  auto products = [&](f32x4 (&st)[4], f32x4 (&pt)[4]) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      st[c] = zero4();
      pt[c] = zero4();
#pragma unroll
      for (int kb = 0; kb < S::KD; ++kb) {
        Frag<T> af;
        load8(af, sk + (16 * c + r) * S::LDH + 32 * kb + 8 * g);
        mma(st[c], af, qf[kb]);
      }
#pragma unroll
      for (int kb = 0; kb < S::KF; ++kb) {
        Frag<T> af;
        load8(af, sf + (16 * c + r) * S::LDF + 32 * kb + 8 * g);
        mma(pt[c], af, ff[kb]);
      }
    }
  };

  // One pass with online rescaling (a row's maximum m changes as tiles arrive; sums
  // taken against the old maximum are multiplied by 2^(m_old - m_new)):
  //   lsum = sum_s 2^(lg_s - m),  wl = sum_s 2^(lg_s - m) log2(pe_s),  den = sum_s P_s,
  // so that CE = -ln 2 wl / lsum + log(den + eps).  lsum, wl and den are partial per lane
  // (its 16 keys of a tile) against the row's common maximum, added across the row's
  // four lane groups when a total is needed.  The gradient
  //   dphi(q_t) = (1/N) (z_t / (den + eps) - acc / lsum),  acc = sum_s 2^(lg_s - m) / pe_s phi(k_s),
  // with z_t the sum of phi(k_s) over the visible keys: every key tile but the last is
  // wholly visible to all 64 queries (the last is the causal diagonal or the ragged end),
  // so those are summed per feature column by the threads (thread: 8 features of DF / 32
  // rows) and enter acc as above; the last tile, where m, lsum and den become final,
  // enters with its complete coefficient G_ts (visible keys only) after acc has been
  // scaled by -(1/N) / lsum.
  float m = -1e30f, lsum = 0.0f, wl = 0.0f, den = 0.0f;
  f32x4 acc[S::NFO];
#pragma unroll
  for (int fo = 0; fo < S::NFO; ++fo) acc[fo] = zero4();
  constexpr int FC = DF / 8, RG = DF / 32;  // 16-byte feature chunks per row; rows per thread
  float zc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) zc[e] = 0.0f;
  const int zf = tid % FC, zr = (tid / FC) * RG;
  TileRows<T, DH, S::LDH, DF, S::LDF> rows_in;
  for (int kt = 0; kt <= last; ++kt) {
    rows_in.load(Kh, Fk, (int64_t)kt * 64, n, tid);  // in flight while the workgroup meets
    __syncthreads();
    rows_in.store(sk, sf, tid);
    __syncthreads();
    f32x4 st[4], pt[4];
    products(st, pt);
    const bool final_tile = kt == last;
    if (GRAD && !final_tile) {  // column sums of a wholly visible tile
#pragma unroll
      for (int rr = 0; rr < RG; ++rr) {
        Frag<T> v;
        load8(v, sf + (zr + rr) * S::LDF + 8 * zf);
#pragma unroll
        for (int e = 0; e < 8; ++e) zc[e] += v.get(e);
      }
    }
    // Keys 64 kt + [0, lim) are visible to this lane's query.  Every tile before the
    // causal diagonal and the ragged end is wholly visible (the test is the same for the
    // whole workgroup): its scores skip the masks.
    const bool whole = (int64_t)kt * 64 + 64 <= n && (!a.causal || kt < qt);
    int lim = 64;
    if (!whole) {
      int64_t l = n - (int64_t)kt * 64;
      if (a.causal) l = l < tq - (int64_t)kt * 64 + 1 ? l : tq - (int64_t)kt * 64 + 1;
      lim = q_ok ? (int)(l < 0 ? 0 : (l > 64 ? 64 : l)) : 0;
    }
    float rescale;
    float cv[4][4];  // gradients: this tile's coefficients of acc (not the final tile)
    auto score = [&](auto whole_tag) {
      constexpr bool W = decltype(whole_tag)::value;
      float tmax = -INFINITY;  // the largest visible score (scale > 0: max commutes with it)
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int j = 0; j < 4; ++j) tmax = fmaxf(tmax, W || 16 * c + 4 * g + j < lim ? st[c][j] : -INFINITY);
      tmax *= c2;
      tmax = fmaxf(tmax, __shfl_xor(tmax, 16, kWave));
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32, kWave));
      const float mn = fmaxf(m, tmax);
      rescale = ex2(m - mn);
      m = mn;
      float add = 0.0f, addw = 0.0f;
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float e = ex2(fmaf(st[c][j], c2, -mn));
          const float pe = pt[c][j] + eps_nt;
          if constexpr (W) {
            add += e;
            addw = fmaf(e, lg2(pe), addw);
            den += pt[c][j];
            if constexpr (GRAD) cv[c][j] = e * rcp(pe);
          } else {  // the same operations, kept only where visible (both paths round alike)
            const bool ok = 16 * c + 4 * g + j < lim;
            add = ok ? add + e : add;
            addw = ok ? fmaf(e, lg2(pe), addw) : addw;
            den = ok ? den + pt[c][j] : den;
            if constexpr (GRAD) cv[c][j] = ok ? e * rcp(pe) : 0.0f;
          }
        }
      lsum = lsum * rescale + add;
      wl = wl * rescale + addw;
    };
    if (!(GRAD && DF == 256) && whole) score(Whole<true>{});  // (one path where registers are tight)
    else score(Whole<false>{});
    if constexpr (GRAD) {
      float fj[4];  // the factors of acc's rows 4 g + j
      if (!final_tile) {
#pragma unroll
        for (int j = 0; j < 4; ++j) fj[j] = __shfl(rescale, 4 * g + j, kWave);
      } else {
        float lt = lsum + __shfl_xor(lsum, 16, kWave);
        lt += __shfl_xor(lt, 32, kWave);
        float dt = den + __shfl_xor(den, 16, kWave);
        dt += __shfl_xor(dt, 32, kWave);
        const float inv_lt = 1.0f / lt, inv_dt = 1.0f / (dt + a.eps);
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            cv[c][j] = 16 * c + 4 * g + j < lim ? a.inv_rows * (inv_dt - cv[c][j] * inv_lt) : 0.0f;
#pragma unroll
        for (int j = 0; j < 4; ++j) fj[j] = -a.inv_rows * __shfl(rescale * inv_lt, 4 * g + j, kWave);
      }
#pragma unroll
      for (int fo = 0; fo < S::NFO; ++fo)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[fo][j] *= fj[j];
#pragma unroll
      for (int kb2 = 0; kb2 < 2; ++kb2) {
        GFrag<T> gf;
        gf.set(cv[2 * kb2], cv[2 * kb2 + 1]);
#pragma unroll
        for (int fo = 0; fo < S::NFO; ++fo) {
          Frag<T> bf;
          load_tr4(bf, 0, sf, S::LDF, 32 * kb2 + 4 * g, 16 * fo, lane);
          load_tr4(bf, 4, sf, S::LDF, 32 * kb2 + 16 + 4 * g, 16 * fo, lane);
          gf.apply(acc[fo], bf);
        }
      }
    }
  }
  lsum += __shfl_xor(lsum, 16, kWave);
  lsum += __shfl_xor(lsum, 32, kWave);
  wl += __shfl_xor(wl, 16, kWave);
  wl += __shfl_xor(wl, 32, kWave);
  den += __shfl_xor(den, 16, kWave);
  den += __shfl_xor(den, 32, kWave);
  if (q_ok && g == 0) {
    const int64_t row = head * n + tq;
    a.row_loss[row] = -kLn2 * wl / lsum + logf(den + a.eps);
    *reinterpret_cast<float4*>(a.stats + row * 4) = float4{m, lsum, den, 0.0f};
  }
  if constexpr (GRAD) {
    // z of the wholly visible tiles: the threads' column sums added over their row groups
    __syncthreads();
    static_assert((64 / RG) * DF * sizeof(float) <= sizeof(sf), "column sums must fit in the feature tile");
    float* zs = reinterpret_cast<float*>(sf);  // [64 / RG][DF] floats in the feature tile (free now)
#pragma unroll
    for (int e = 0; e < 8; ++e) zs[(zr / RG) * DF + 8 * zf + e] = zc[e];
    __syncthreads();
    float zcoef[4];  // (1/N) / (den + eps) of acc's rows 4 g + j
#pragma unroll
    for (int j = 0; j < 4; ++j) zcoef[j] = a.inv_rows / (__shfl(den, 4 * g + j, kWave) + a.eps);
#pragma unroll
    for (int fo = 0; fo < S::NFO; ++fo) {
      float z = 0.0f;
      for (int q = 0; q < 64 / RG; ++q) z += zs[q * DF + 16 * fo + r];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t t = (int64_t)qt * 64 + wave * 16 + 4 * g + j;
        if (t < n) a.dphiq[(head * n + t) * DF + 16 * fo + r] = acc[fo][j] + zcoef[j] * z;
      }
    }
  }
}

template <typename T, int DH, int DF>
__global__ __launch_bounds__(256, 2) void distill_k_kernel(DistillArgs a) {
  using S = DistShape<T, DH, DF>;
  __shared__ __align__(16) T sq[64 * S::LDH];
  __shared__ __align__(16) T sf[64 * S::LDF];
  __shared__ __align__(16) float sst[64 * 4];
  const int tid = threadIdx.x, wave = wave_id(), lane = tid % kWave;
  const int g = lane / 16, r = lane % 16;
  const int64_t n = a.n;
  const int ntiles = (int)((n + 63) / 64);
  const int64_t item = xcd_item(blockIdx.x, gridDim.x);
  const int64_t head = item / ntiles;
  const int kt = (int)(item - head * ntiles);
  const int64_t tk = (int64_t)kt * 64 + wave * 16 + r;  // this lane's key
  const bool k_ok = tk < n;
  const T* Qh = reinterpret_cast<const T*>(a.Q) + head * n * DH;
  const T* Fq = reinterpret_cast<const T*>(a.phiq) + head * n * DF;
  const float* st_h = a.stats + head * n * 4;
  Frag<T> kf[S::KD], ff[S::KF];
  {
    const T* k = reinterpret_cast<const T*>(a.K) + (head * n + (k_ok ? tk : 0)) * DH;
    const T* f = reinterpret_cast<const T*>(a.phik) + (head * n + (k_ok ? tk : 0)) * DF;
#pragma unroll
    for (int kb = 0; kb < S::KD; ++kb) {
      if (k_ok) load8(kf[kb], k + 32 * kb + 8 * g);
      else kf[kb].zero();
    }
#pragma unroll
    for (int kb = 0; kb < S::KF; ++kb) {
      if (k_ok) load8(ff[kb], f + 32 * kb + 8 * g);
      else ff[kb].zero();
    }
  }
  const float c2 = a.scale * kLog2e;
  f32x4 dk[S::NFO];
#pragma unroll
  for (int fo = 0; fo < S::NFO; ++fo) dk[fo] = zero4();
  TileRows<T, DH, S::LDH, DF, S::LDF> rows_in;
  for (int qt = a.causal ? kt : 0; qt < ntiles; ++qt) {
    // the tile's reads (rows and, threads 0..63, the query statistics m, lsum, den)
    // before the barrier that frees the tiles
    rows_in.load(Qh, Fq, (int64_t)qt * 64, n, tid);
    const int64_t q = (int64_t)qt * 64 + tid;
    float4 sv = float4{0.0f, 1.0f, 0.0f, 0.0f};
    if (tid < 64 && q < n) sv = *reinterpret_cast<const float4*>(st_h + q * 4);
    __syncthreads();
    rows_in.store(sq, sf, tid);
    if (tid < 64)  // per query: m, 1 / lsum, 1 / (den + eps), eps / n_t (zeros past n: never visible)
      *reinterpret_cast<float4*>(sst + 4 * tid) =
          q < n ? float4{sv.x, 1.0f / sv.y, 1.0f / (sv.z + a.eps), a.eps / (float)(a.causal ? q + 1 : n)}
                : float4{0.0f, 0.0f, 0.0f, 1.0f};
    __syncthreads();
    // Queries 64 qt + [qlo, qhi) see this lane's key; a tile before the ragged end and
    // (causal) past the diagonal is seen whole by every key of the workgroup.
    const bool whole = (int64_t)qt * 64 + 64 <= n && (!a.causal || qt > kt);
    int qlo = 0, qhi = 64;
    if (!whole) {
      const int64_t hi = n - (int64_t)qt * 64;
      qhi = k_ok ? (int)(hi > 64 ? 64 : hi) : 0;
      if (a.causal) {
        const int64_t lo = tk - (int64_t)qt * 64;
        qlo = (int)(lo < 0 ? 0 : (lo > 64 ? 64 : lo));
      }
    }
    // S and P of query tile qt: s[c][j], p[c][j] for query 64 qt + 16 c + 4 g + j
    float gv[4][4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      f32x4 s = zero4(), p = zero4();
#pragma unroll
      for (int kb = 0; kb < S::KD; ++kb) {
        Frag<T> af;
        load8(af, sq + (16 * c + r) * S::LDH + 32 * kb + 8 * g);
        mma(s, af, kf[kb]);
      }
#pragma unroll
      for (int kb = 0; kb < S::KF; ++kb) {
        Frag<T> af;
        load8(af, sf + (16 * c + r) * S::LDF + 32 * kb + 8 * g);
        mma(p, af, ff[kb]);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int qi = 16 * c + 4 * g + j;
        const float4 sv = *reinterpret_cast<const float4*>(sst + 4 * qi);
        const float A = ex2(fmaf(s[j], c2, -sv.x)) * sv.y;
        const float gval = a.inv_rows * (sv.z - A * rcp(p[j] + sv.w));
        gv[c][j] = whole || (qi >= qlo && qi < qhi) ? gval : 0.0f;
      }
    }
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2) {
      GFrag<T> gf;
      gf.set(gv[2 * kb2], gv[2 * kb2 + 1]);
#pragma unroll
      for (int fo = 0; fo < S::NFO; ++fo) {
        Frag<T> bf;
        load_tr4(bf, 0, sf, S::LDF, 32 * kb2 + 4 * g, 16 * fo, lane);
        load_tr4(bf, 4, sf, S::LDF, 32 * kb2 + 16 + 4 * g, 16 * fo, lane);
        gf.apply(dk[fo], bf);
      }
    }
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t s = (int64_t)kt * 64 + wave * 16 + 4 * g + j;
    if (s < n) {
      float* o = a.dphik + (head * n + s) * DF + r;
#pragma unroll
      for (int fo = 0; fo < S::NFO; ++fo) o[16 * fo] = dk[fo][j];
    }
  }
}

template <typename T, int DH, int DF>
hipError_t distill_launch(const DistillArgs& a, bool grads, hipStream_t s) {
  const int64_t items = a.heads * ((a.n + 63) / 64);
  if (grads) {
    hipLaunchKernelGGL((distill_q_kernel<T, DH, DF, true>), dim3((unsigned)items), dim3(256), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((distill_k_kernel<T, DH, DF>), dim3((unsigned)items), dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL((distill_q_kernel<T, DH, DF, false>), dim3((unsigned)items), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

template <typename T, int DH>
hipError_t distill_dispatch_D(int D, const DistillArgs& a, bool grads, hipStream_t s) {
  switch (D) {
    case 64: return distill_launch<T, DH, 64>(a, grads, s);
    case 128: return distill_launch<T, DH, 128>(a, grads, s);
    case 256:
      if constexpr (sizeof(T) == 2) return distill_launch<T, DH, 256>(a, grads, s);
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
}

template <typename T>
hipError_t distill_dispatch(int d, int D, const DistillArgs& a, bool grads, hipStream_t s) {
  switch (d) {
    case 32: return distill_dispatch_D<T, 32>(D, a, grads, s);
    case 64: return distill_dispatch_D<T, 64>(D, a, grads, s);
    case 128: return distill_dispatch_D<T, 128>(D, a, grads, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

bool distill_supported(Dt dt, int d, int D) {
  if (d != 32 && d != 64 && d != 128) return false;
  return D == 64 || D == 128 || (D == 256 && dt == Dt::BF16);
}

hipError_t launch_distill(Dt dt, int d, int D, const DistillArgs& a, bool grads, hipStream_t s) {
  if (!distill_supported(dt, d, D)) return hipErrorInvalidValue;
  return dt == Dt::BF16 ? distill_dispatch<__bf16>(d, D, a, grads, s) : distill_dispatch<float>(d, D, a, grads, s);
}

}  // namespace luna
