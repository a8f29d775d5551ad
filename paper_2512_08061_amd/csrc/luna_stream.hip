// luna_stream.hip -- one streaming step of causal LUNA attention: the prefix form of
// eq. (9) of Section 3.1 continued from a given state (S, z) over m new tokens,
//
//   for t = 0 .. m - 1:  S += phi(k_t) v_t^T,  z += phi(k_t),
//                        out_t = phi(q_t)^T S / (phi(q_t)^T z + eps),
//
// the recurrent form of the runtime section (section 4).  The features of the new
// queries and keys come from the feature-map kernel (fp32); this kernel carries the
// state.
//
// One workgroup per (head, block of 32 value columns).  Thread (g, q) holds, for the
// features f = g + 32 i of its group g (i < 8; interleaved, so that the groups of a
// wave read consecutive LDS words of a feature row), the four columns 4q .. 4q + 3 of
// S as float4 and the same features of z, in fp32 registers for the whole step.  Per
// token it adds the key's outer product and forms its partial numerator (four
// columns) and denominator; the eight groups of a wave are added across lanes on the VALU
// and the four waves through LDS, in a fixed order (deterministic), for all of a
// stage's tokens after one barrier, so that the tokens' shuffles overlap the next
// tokens' updates.  The state is read once at the start and written once at the end (16-byte
// accesses), so a step of m tokens costs one pass over S whatever m is.  z is read
// from a copy that the feature-map launch takes: the column blocks of a head are not
// ordered against one another, and block 0 writes the new z in place.
#include "luna_device.hpp"
#include "luna_kernels.hpp"

namespace luna {

namespace {

constexpr int kStepCols = 32;                       // value columns per workgroup
constexpr int kStepQuads = kStepCols / 4;           // column quads per workgroup
constexpr int kStepGroups = 256 / kStepQuads;       // feature groups
constexpr int kStepFeat = kStepMaxD / kStepGroups;  // features per thread
constexpr int kStepTokens = 16;                     // tokens staged in LDS at a time
constexpr int kStepMfmaMinTokens = 16;              // steps this long run on the matrix cores
static_assert(kStepMaxD == 256, "one thread per feature row of the staged tokens");
static_assert(kStepTokens * kStepCols % 256 == 0, "whole value entries per thread");

// x plus the x of lane l ^ 8, ^ 16 and ^ 32, on the VALU: a rotation by 8 within each
// row of 16 lanes (data-parallel primitive) pairs lane l with l ^ 8; a permlane swap of a
// value with itself leaves every lane its own value in one result and its partner's in
// the other.  Each step adds a pair of values, so both lanes of a pair get the same sum.
__device__ __forceinline__ float step_sum_xor8(float x) {
  return x + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x128, 0xf, 0xf, true));
}
__device__ __forceinline__ float step_sum_xor16(float x) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}
__device__ __forceinline__ float step_sum_xor32(float x) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}
__device__ __forceinline__ float step_sum_groups(float x) {
  static_assert(kStepQuads == 8, "the groups of a wave are lane bits 3..5");
  return step_sum_xor32(step_sum_xor16(step_sum_xor8(x)));
}

template <typename T>
__global__ __launch_bounds__(256) void causal_step_kernel(StepArgs a) {
  __shared__ float sq[kStepTokens][kStepMaxD];
  __shared__ float sk[kStepTokens][kStepMaxD];
  __shared__ __attribute__((aligned(16))) float sv[kStepTokens][kStepCols];
  __shared__ float red[kStepTokens][4][kStepQuads][5];  // per token, wave and column quad: four numerators, the denominator

  const int nblk = a.d / kStepCols;
  const int head = blockIdx.x / nblk;
  const int cblk = blockIdx.x - head * nblk;
  const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
  const int q = tid % kStepQuads, grp = tid / kStepQuads;
  const int D = a.D, d = a.d, m = a.m;
  const int col0 = cblk * kStepCols + 4 * q;
  float* S = a.S + (size_t)head * D * d;
  float* z = a.z + (size_t)head * D;
  const float* z0 = a.z_in + (size_t)head * D;
  const float* PQ = a.phiq + (size_t)head * m * D;
  const float* PK = a.phik + (size_t)head * m * D;
  const T* V = reinterpret_cast<const T*>(a.V) + (size_t)head * m * d;
  T* out = reinterpret_cast<T*>(a.out) + (size_t)head * m * d;

  float4 s[kStepFeat];
  float zz[kStepFeat];
#pragma unroll
  for (int i = 0; i < kStepFeat; ++i) {
    const int f = grp + kStepGroups * i;
    s[i] = f < D ? *reinterpret_cast<const float4*>(&S[(size_t)f * d + col0]) : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    zz[i] = f < D ? z0[f] : 0.0f;
  }

  for (int t0 = 0; t0 < m; t0 += kStepTokens) {
    const int tn = min(kStepTokens, m - t0);
    // thread tid stages feature tid of every token of the stage (features past D and
    // tokens past the step as zeros) and two value entries; all loads are issued
    // before the first store, so that their latencies overlap
    float rq[kStepTokens], rk[kStepTokens], rv[kStepTokens * kStepCols / 256];
#pragma unroll
    for (int tt = 0; tt < kStepTokens; ++tt) {
      const bool ok = tt < tn && tid < D;
      rq[tt] = ok ? PQ[(size_t)(t0 + tt) * D + tid] : 0.0f;
      rk[tt] = ok ? PK[(size_t)(t0 + tt) * D + tid] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < kStepTokens * kStepCols / 256; ++j) {
      const int tt = tid / kStepCols + (256 / kStepCols) * j, c = tid % kStepCols;
      rv[j] = tt < tn ? (float)V[(size_t)(t0 + tt) * d + cblk * kStepCols + c] : 0.0f;
    }
    __syncthreads();  // the previous stage's tokens are no longer read
#pragma unroll
    for (int tt = 0; tt < kStepTokens; ++tt) {
      sq[tt][tid] = rq[tt];
      sk[tt][tid] = rk[tt];
    }
#pragma unroll
    for (int j = 0; j < kStepTokens * kStepCols / 256; ++j)
      sv[tid / kStepCols + (256 / kStepCols) * j][tid % kStepCols] = rv[j];
    __syncthreads();
#pragma unroll
    for (int tt = 0; tt < kStepTokens; ++tt) {
      if (tt < tn) {  // (uniform)
        const float4 v = *reinterpret_cast<const float4*>(&sv[tt][4 * q]);
        float4 num = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        float den = 0.0f;
#pragma unroll
        for (int i = 0; i < kStepFeat; ++i) {
          const int f = grp + kStepGroups * i;
          const float kf = sk[tt][f], qf = sq[tt][f];
          s[i].x = fmaf(kf, v.x, s[i].x);
          s[i].y = fmaf(kf, v.y, s[i].y);
          s[i].z = fmaf(kf, v.z, s[i].z);
          s[i].w = fmaf(kf, v.w, s[i].w);
          zz[i] += kf;
          num.x = fmaf(qf, s[i].x, num.x);
          num.y = fmaf(qf, s[i].y, num.y);
          num.z = fmaf(qf, s[i].z, num.z);
          num.w = fmaf(qf, s[i].w, num.w);
          den = fmaf(qf, zz[i], den);
        }
        // the eight groups of this wave (lane bits 3..5)
        num.x = step_sum_groups(num.x);
        num.y = step_sum_groups(num.y);
        num.z = step_sum_groups(num.z);
        num.w = step_sum_groups(num.w);
        den = step_sum_groups(den);
        if (lane < kStepQuads) {
          red[tt][wave][q][0] = num.x;
          red[tt][wave][q][1] = num.y;
          red[tt][wave][q][2] = num.z;
          red[tt][wave][q][3] = num.w;
          red[tt][wave][q][4] = den;
        }
      }
    }
    // the four waves of every staged token at once: one barrier per stage, not per token
    __syncthreads();
    for (int idx = tid; idx < tn * kStepCols; idx += blockDim.x) {
      const int tt = idx / kStepCols, c = idx % kStepCols;
      float nu = 0.0f, de = 0.0f;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        nu += red[tt][w][c / 4][c % 4];
        de += red[tt][w][c / 4][4];
      }
      out[(size_t)(t0 + tt) * d + cblk * kStepCols + c] = (T)(nu / (de + a.eps));
    }
  }

#pragma unroll
  for (int i = 0; i < kStepFeat; ++i) {
    const int f = grp + kStepGroups * i;
    if (f < D) {
      *reinterpret_cast<float4*>(&S[(size_t)f * d + col0]) = s[i];
      if (cblk == 0 && q == 0) z[f] = zz[i];  // every column block carries the same z
    }
  }
}

// The same step for longer steps, on the matrix cores in fp32 (v_mfma_f32_16x16x4_f32):
// per stage of 16 tokens, in the chunked form of the prefix sums,
//
//   out = (phi(Q) S + mask(phi(Q) phi(K)^T) V) / (phi(Q) z + mask(phi(Q) phi(K)^T) 1 + eps),
//   S += phi(K)^T V,  z += phi(K)^T 1,
//
// with S and z the state before the stage and mask keeping key <= query.  Wave w holds
// the rows 64w .. 64w + 63 of S (four 16-feature tiles by the workgroup's two 16-column
// tiles) and of z (as a tile of 16 equal columns) as accumulator tiles: lane (g, c) holds
// features 16t + 4g + j, column c.  The readout contracts over features in the order
// that makes those registers its B operand as they are (k-slot g of k-step j is feature
// 16t + 4g + j); the update contracts over tokens and writes the same tiles.  Each wave
// forms its features' share of the readout and of the 16 x 16 scores; the shares are
// added through LDS in a fixed order, and waves 0 and 1 finish one column tile each.
constexpr int kStepRow = kStepMaxD + 4;  // padded LDS row of a staged token's features

template <typename T>
__global__ __launch_bounds__(256) void causal_step_mfma_kernel(StepArgs a) {
  // the staged tokens' features; before the first stage and after the last they hold
  // the workgroup's S columns [feature][32], 16-byte chunks swapped between the two
  // column halves on every other group of four rows (two lane groups of an accumulator
  // read then hit different banks)
  __shared__ __attribute__((aligned(16))) float sqk[2][kStepTokens][kStepRow];
  static_assert(2 * kStepTokens * kStepRow >= kStepMaxD * kStepCols, "S columns fit the token buffers");
  float (&sq)[kStepTokens][kStepRow] = sqk[0];
  float (&sk)[kStepTokens][kStepRow] = sqk[1];
  float* const st = &sqk[0][0][0];
  auto st_at = [](int f, int col) { return f * kStepCols + (col ^ (16 * ((f >> 2) & 1))); };
  __shared__ float sv[kStepTokens][kStepCols];
  __shared__ float rnum[4][kStepTokens][kStepCols + 1];     // per wave: readout numerators
  __shared__ float rden[4][kStepTokens];                    // per wave: phi(q) . z
  __shared__ float rsc[4][kStepTokens][kStepTokens + 1];    // per wave: scores [key][query]

  const int nblk = a.d / kStepCols;
  const int head = blockIdx.x / nblk;
  const int cblk = blockIdx.x - head * nblk;
  const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
  const int g = lane / 16, c = lane % 16;
  const int D = a.D, d = a.d, m = a.m;
  const int col0 = cblk * kStepCols;
  const int fw = 64 * wave;  // this wave's first feature
  float* S = a.S + (size_t)head * D * d;
  float* z = a.z + (size_t)head * D;
  const float* z0 = a.z_in + (size_t)head * D;
  const float* PQ = a.phiq + (size_t)head * m * D;
  const float* PK = a.phik + (size_t)head * m * D;
  const T* V = reinterpret_cast<const T*>(a.V) + (size_t)head * m * d;
  T* out = reinterpret_cast<T*>(a.out) + (size_t)head * m * d;

  // S columns into LDS with 16-byte loads (features past D as zeros), then into the
  // accumulator tiles
#pragma unroll
  for (int i = 0; i < kStepMaxD * kStepCols / 4 / 256; ++i) {
    const int idx = tid + 256 * i, f = idx / (kStepCols / 4), q4 = 4 * (idx % (kStepCols / 4));
    const float4 v = f < D ? *reinterpret_cast<const float4*>(&S[(size_t)f * d + col0 + q4])
                           : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    *reinterpret_cast<float4*>(&st[st_at(f, q4)]) = v;
  }
  __syncthreads();
  f32x4 sc[4][2], zc[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int f = fw + 16 * t + 4 * g + j;
      sc[t][0][j] = st[st_at(f, c)];
      sc[t][1][j] = st[st_at(f, 16 + c)];
      zc[t][j] = f < D ? z0[f] : 0.0f;
    }
  }

  for (int t0 = 0; t0 < m; t0 += kStepTokens) {
    const int tn = min(kStepTokens, m - t0);
    // thread tid stages feature tid of every token of the stage (features past D and
    // tokens past the step as zeros, which add nothing below) and two value entries
    float rq[kStepTokens], rk[kStepTokens], rv[kStepTokens * kStepCols / 256];
#pragma unroll
    for (int tt = 0; tt < kStepTokens; ++tt) {
      const bool ok = tt < tn && tid < D;
      rq[tt] = ok ? PQ[(size_t)(t0 + tt) * D + tid] : 0.0f;
      rk[tt] = ok ? PK[(size_t)(t0 + tt) * D + tid] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < kStepTokens * kStepCols / 256; ++j) {
      const int tt = tid / kStepCols + (256 / kStepCols) * j;
      rv[j] = tt < tn ? (float)V[(size_t)(t0 + tt) * d + col0 + tid % kStepCols] : 0.0f;
    }
    __syncthreads();  // the previous stage's tokens and shares are no longer read
#pragma unroll
    for (int tt = 0; tt < kStepTokens; ++tt) {
      sq[tt][tid] = rq[tt];
      sk[tt][tid] = rk[tt];
    }
#pragma unroll
    for (int j = 0; j < kStepTokens * kStepCols / 256; ++j)
      sv[tid / kStepCols + (256 / kStepCols) * j][tid % kStepCols] = rv[j];
    __syncthreads();

    // this wave's features' share of phi(Q) S, phi(Q) z and the scores phi(K) phi(Q)^T,
    // from the state before the stage
    f32x4 np0 = zero4(), np1 = zero4(), dp = zero4(), gp = zero4();
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const float4 qa = *reinterpret_cast<const float4*>(&sq[c][fw + 16 * t + 4 * g]);
      const float4 ka = *reinterpret_cast<const float4*>(&sk[c][fw + 16 * t + 4 * g]);
      const float qv[4] = {qa.x, qa.y, qa.z, qa.w}, kv[4] = {ka.x, ka.y, ka.z, ka.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        np0 = __builtin_amdgcn_mfma_f32_16x16x4f32(qv[j], sc[t][0][j], np0, 0, 0, 0);
        np1 = __builtin_amdgcn_mfma_f32_16x16x4f32(qv[j], sc[t][1][j], np1, 0, 0, 0);
        dp = __builtin_amdgcn_mfma_f32_16x16x4f32(qv[j], zc[t][j], dp, 0, 0, 0);
        gp = __builtin_amdgcn_mfma_f32_16x16x4f32(kv[j], qv[j], gp, 0, 0, 0);
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {  // row 4g + j: a token (readout) or a key (scores)
      rnum[wave][4 * g + j][c] = np0[j];
      rnum[wave][4 * g + j][16 + c] = np1[j];
      rsc[wave][4 * g + j][c] = gp[j];
      if (c == 0) rden[wave][4 * g + j] = dp[j];
    }

    // the stage's keys into the state (k-slot g of k-step j is token 4g + j)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int tk = 4 * g + j;
      const float v0 = sv[tk][c], v1 = sv[tk][16 + c];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const float kf = sk[tk][fw + 16 * t + c];  // A operand: row = feature fw + 16t + c
        sc[t][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(kf, v0, sc[t][0], 0, 0, 0);
        sc[t][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(kf, v1, sc[t][1], 0, 0, 0);
        zc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(kf, 1.0f, zc[t], 0, 0, 0);
      }
    }
    __syncthreads();

    if (wave < 2) {  // (uniform) wave ct finishes column tile ct
      const int ct = wave;
      // the masked scores as A operand (row = query c, k-slot g of k-step j = key 4g + j)
      f32x4 ni = zero4(), di = zero4();
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int key = 4 * g + j;
        float sg = ((rsc[0][key][c] + rsc[1][key][c]) + rsc[2][key][c]) + rsc[3][key][c];
        sg = key <= c ? sg : 0.0f;
        ni = __builtin_amdgcn_mfma_f32_16x16x4f32(sg, sv[key][16 * ct + c], ni, 0, 0, 0);
        di = __builtin_amdgcn_mfma_f32_16x16x4f32(sg, 1.0f, di, 0, 0, 0);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int tt = 4 * g + j;  // C row: token
        if (tt < tn) {
          const int col = 16 * ct + c;
          const float nu = ((rnum[0][tt][col] + rnum[1][tt][col]) + (rnum[2][tt][col] + rnum[3][tt][col])) + ni[j];
          const float de = ((rden[0][tt] + rden[1][tt]) + (rden[2][tt] + rden[3][tt])) + di[j];
          out[(size_t)(t0 + tt) * d + col0 + col] = (T)(nu / (de + a.eps));
        }
      }
    }
  }

  // the accumulator tiles back through LDS (no wave reads the token buffers after the
  // last stage's update), then 16-byte stores of the rows below D
#pragma unroll
  for (int t = 0; t < 4; ++t) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int f = fw + 16 * t + 4 * g + j;
      st[st_at(f, c)] = sc[t][0][j];
      st[st_at(f, 16 + c)] = sc[t][1][j];
      if (f < D && cblk == 0 && c == 0) z[f] = zc[t][j];  // every column block carries the same z
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kStepMaxD * kStepCols / 4 / 256; ++i) {
    const int idx = tid + 256 * i, f = idx / (kStepCols / 4), q4 = 4 * (idx % (kStepCols / 4));
    if (f < D) *reinterpret_cast<float4*>(&S[(size_t)f * d + col0 + q4]) = *reinterpret_cast<const float4*>(&st[st_at(f, q4)]);
  }
}

}  // namespace

hipError_t launch_causal_step(Dt dt, const StepArgs& a, hipStream_t s) {
  if (a.d % kStepCols != 0 || a.D > kStepMaxD) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(a.heads * (a.d / kStepCols)));
  const bool mfma = a.m >= kStepMfmaMinTokens;
  if (dt == Dt::BF16) {
    if (mfma) hipLaunchKernelGGL(causal_step_mfma_kernel<__bf16>, grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL(causal_step_kernel<__bf16>, grid, dim3(256), 0, s, a);
  } else {
    if (mfma) hipLaunchKernelGGL(causal_step_mfma_kernel<float>, grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL(causal_step_kernel<float>, grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace luna
