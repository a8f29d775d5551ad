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

template <typename T, int DH, int DF>
struct DistShape {
  static constexpr int PAD = 16 / (int)sizeof(T);  // one 16-byte chunk per row
  static constexpr int LDH = DH + PAD, LDF = DF + PAD;
  static constexpr int KD = DH / 32, KF = DF / 32, NFO = DF / 16;
};

// Rows r0 .. r0 + 63 of a row-major [n][W] array of T into an LDS tile with row stride
// LD (rows at or past n as zeros), 16 bytes per thread and step.
template <typename T, int W, int LD>
__device__ __forceinline__ void stage_rows(T* tile, const T* src, int64_t r0, int64_t n, int tid) {
  constexpr int CH = W * (int)sizeof(T) / 16;
  for (int i = tid; i < 64 * CH; i += 256) {
    const int row = i / CH, c = i % CH;
    uint4 v = {0u, 0u, 0u, 0u};
    if (r0 + row < n) v = *reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(src + (r0 + row) * W) + 16 * c);
    *reinterpret_cast<uint4*>(reinterpret_cast<char*>(tile + row * LD) + 16 * c) = v;
  }
}

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

template <typename T, int DH, int DF, bool GRAD>
__global__ __launch_bounds__(256, 2) void distill_q_kernel(DistillArgs a) {
  using S = DistShape<T, DH, DF>;
  __shared__ __align__(16) T sk[64 * S::LDH];
  __shared__ __align__(16) T sf[64 * S::LDF];
  const int tid = threadIdx.x, wave = wave_id(), lane = tid % kWave;
  const int g = lane / 16, r = lane % 16;
  const int64_t n = a.n;
  const int ntiles = (int)((n + 63) / 64);
  const int64_t head = blockIdx.x / ntiles;
  // causal: the last query tiles (the most key tiles) are dispatched first
  const int qt = a.causal ? ntiles - 1 - (int)(blockIdx.x - head * ntiles) : (int)(blockIdx.x - head * ntiles);
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
  auto stage = [&](int kt) {
    __syncthreads();
    stage_rows<T, DH, S::LDH>(sk, Kh, (int64_t)kt * 64, n, tid);
    stage_rows<T, DF, S::LDF>(sf, Fk, (int64_t)kt * 64, n, tid);
    __syncthreads();
  };
  auto visible = [&](int kt, int c, int j) {
    const int64_t s = (int64_t)kt * 64 + 16 * c + 4 * g + j;
    return q_ok && s < n && (!a.causal || s <= tq);
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
  for (int kt = 0; kt <= last; ++kt) {
    stage(kt);
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
    float lg[4][4], tmax = -INFINITY;
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        lg[c][j] = visible(kt, c, j) ? st[c][j] * c2 : -INFINITY;
        tmax = fmaxf(tmax, lg[c][j]);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, kWave));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, kWave));
    const float mn = fmaxf(m, tmax);
    const float rescale = exp2f(m - mn);
    m = mn;
    float add = 0.0f, addw = 0.0f;
    float cv[4][4];  // gradients: this tile's coefficients of acc (not the final tile)
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bool ok = lg[c][j] != -INFINITY;
        const float e = exp2f(lg[c][j] - mn);
        const float pe = pt[c][j] + eps_nt;
        add += e;
        addw += ok ? e * log2f(pe) : 0.0f;
        if (ok) den += pt[c][j];
        cv[c][j] = e / pe;  // 0 where masked (e = 0)
      }
    lsum = lsum * rescale + add;
    wl = wl * rescale + addw;
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
            cv[c][j] = lg[c][j] != -INFINITY ? a.inv_rows * (inv_dt - cv[c][j] * inv_lt) : 0.0f;
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
  const int64_t head = blockIdx.x / ntiles;
  const int kt = (int)(blockIdx.x - head * ntiles);
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
  for (int qt = a.causal ? kt : 0; qt < ntiles; ++qt) {
    __syncthreads();
    stage_rows<T, DH, S::LDH>(sq, Qh, (int64_t)qt * 64, n, tid);
    stage_rows<T, DF, S::LDF>(sf, Fq, (int64_t)qt * 64, n, tid);
    if (tid < 64) {
      const int64_t q = (int64_t)qt * 64 + tid;
      *reinterpret_cast<float4*>(sst + 4 * tid) =
          q < n ? *reinterpret_cast<const float4*>(st_h + q * 4) : float4{0.0f, 1.0f, 0.0f, 0.0f};
    }
    __syncthreads();
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
        const int64_t q = (int64_t)qt * 64 + qi;
        gv[c][j] = 0.0f;
        if (k_ok && q < n && (!a.causal || tk <= q)) {
          const float4 sv = *reinterpret_cast<const float4*>(sst + 4 * qi);  // m, sum, den
          const float A = exp2f(s[j] * c2 - sv.x) / sv.y;
          const float pe = p[j] + a.eps / (float)(a.causal ? q + 1 : n);
          gv[c][j] = a.inv_rows * (1.0f / (sv.z + a.eps) - A / pe);
        }
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
