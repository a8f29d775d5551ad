// luna_causal.hip -- causal (streaming) LUNA attention as a chunked prefix scan.
//
// out_t = phi(q_t)^T S_t / (phi(q_t)^T z_t + eps) with S_t, z_t summed over s <= t.
// Tokens are processed in chunks of 64; within chunk c (query rows t, key columns s):
//
//   P      = tril(phi(Q_c) phi(K_c)^T)              (diagonal included)
//   num    = P V_c + phi(Q_c) S_{c-1},   den = P 1 + phi(Q_c) z_{c-1}
//   S_c    = S_{c-1} + phi(K_c)^T V_c,   z_c = z_{c-1} + phi(K_c)^T 1
//
// which regroups the prefix sums exactly.
//
// Work split.  One workgroup owns one (head, part of the sequence).  With few heads
// a head's tokens are cut in two at a chunk boundary x: part 0 scans [0, x) from a
// zero state; part 1 first accumulates the state of [0, x) (keys and values only,
// no readout) and then scans [x, n).  The cut is placed so that both parts take
// about the same time; nothing is shared between workgroups.
//
// Roles.  Eight waves, two per SIMD: four matrix waves and four map waves, so that
// every SIMD pairs matrix-core work with vector and table-lookup work.
//  - Map wave p computes phi of query rows 16p .. 16p + 15 and key rows
//    16p .. 16p + 15 of the next chunk (projection on the matrix cores, the
//    piecewise-linear channel functions in registers) and stages V; phi(Q) is
//    stored token-major and phi(K) feature-major in LDS.
//  - Matrix wave m owns value columns 32m .. 32m + 31 (d / 4 of them) and keeps
//    that slice of S (all features) in fp32 accumulators.  It forms its share of
//    the P^T blocks and of phi(Q_c) z_{c-1}, then num^T = S_{c-1}^T phi(Q_c)^T with
//    S taken straight from the accumulators (the feature order of S's rows makes
//    two accumulator tiles one k-fragment of S^T), then num^T += V^T P^T, the
//    division and the store, then S += phi(K_c)^T V_c and z += phi(K_c)^T 1.
// Per chunk c, three barriers:
//   B1: phi(Q_c), phi(K_c), V_c, z_{c-1} in LDS.
//       matrix: P^T blocks, phi(Q_c) z_{c-1}, readout.   map: phi(Q_{c+1}) to registers.
//   B2: P and den parts in LDS; phi(Q_c) no longer read.
//       matrix: P V, output, state update.
//       map: phi(Q_{c+1}) to LDS, z_c published, phi(K_{c+1}) to registers.
//   B3: phi(K_c), V_c no longer read.   map: phi(K_{c+1}), V_{c+1} to LDS.
// Large operands are one 16-byte LDS read per lane; only the P^T blocks (phi(K)
// columns) and V use the gfx950 transpose read.  Q, K and V rows are fetched one
// chunk ahead.
#include "luna_device.hpp"
#include "luna_kernels.hpp"

namespace luna {

template <typename T, int DH, int L, int MB>
struct CsCfg {
  static constexpr int NCB = DH / 16;                 // 16-column blocks of the value width
  static constexpr int CBW = NCB >= 4 ? NCB / 4 : 1;  // column blocks per matrix wave
  static constexpr int NMW = NCB / CBW;               // matrix waves that own columns (2 or 4)
  static constexpr int KS = DH / 32;                  // 32-wide k-steps of the projection
  static constexpr int FP = 16 * MB * L;              // features, projections padded to 16
  static constexpr int NF = FP / 32;                  // 32-feature k-fragments
  static constexpr int RB = FP / 16;                  // 16-feature row blocks of S
  static constexpr int NDEN = 4 / NMW;                // query blocks whose phi(Q) z a matrix wave forms
  static constexpr int VE = 16 / (int)sizeof(T);      // elements per 16-byte chunk
  static constexpr int NPQ = MB * 4 * L / 8;          // phi(Q) fragments per lane per block
  static constexpr int NPK = MB * L / 2;              // phi(K) fragments (two channels x four tokens)
  static constexpr int VPT = 64 * DH / VE / 256;      // 16-byte V chunks per map-wave thread
  static constexpr int NSEG = nseg_cap(L, kAttnSegBytes);
  static_assert(NCB == 2 || NCB == 4 || NCB == 8, "d must be 32, 64 or 128");
  static_assert(FP % 32 == 0 && L % 2 == 0, "features must fill 32-wide fragments");
};

template <typename T, int DH, int L, int MB>
struct CsLds {
  using C = CsCfg<T, DH, L, MB>;
  typename PwlTab<T, L, C::NSEG>::type tab;
  alignas(16) T wfr[MB][C::KS][kWave][8];  // W fragments (A of u^T = W X^T, B of u = X W^T)
  alignas(16) T phq[64 * C::FP];           // phi(Q_c), token-major
  alignas(16) T phk[C::FP * 64];           // phi(K_c)^T, feature-major
  alignas(16) T pm[64 * 64];               // P, query-major (blocks above the diagonal stay 0)
  alignas(16) T vt[64 * DH];               // V_c, token-major
  alignas(16) float denp[4][64];           // row sums of P per key block
  alignas(16) float deni[64];              // phi(Q_c) z_{c-1}
  alignas(16) float zp[4][C::FP];          // z_c over each map wave's key rows
  alignas(16) float zs[2][C::FP];          // z_c, summed, by chunk parity
  float bias[16 * MB];                     // projection biases, 0 for padded projections
};

// 16-byte chunk swizzles: physical chunk of logical chunk `cg` in row `row` of a
// tile with CPR chunks per row.
// phi(Q) and P: the 16 consecutive rows one read touches land on 16 distinct
// chunk slots of a 256-byte bank window.
template <int CPR>
__device__ __forceinline__ int swz_rows16(int row, int cg) {
  if constexpr (CPR >= 16) return cg ^ (row & 15);
  else return cg ^ ((row / (16 / CPR)) & (CPR - 1));
}
// phi(K)^T: read in the row order of s_feature (below): 16 rows that differ in
// bits 0, 1, 3 and 4; written by 16 lanes whose rows differ in bits 3 to 6.
template <int CPR>
__device__ __forceinline__ int swz_k(int row, int cg) {
  const int b = [&] {
    if constexpr (CPR >= 16) return (row & 3) | ((row >> 1) & 12);
    else return (((row >> 1) ^ (row >> 5)) & 1) | ((((row >> 3) ^ (row >> 6)) & 1) << 1) | (((row >> 4) & 1) << 2);
  }();
  return cg ^ b;
}
// V: transpose reads of four (and eight) consecutive rows.
template <int CPR>
__device__ __forceinline__ int swz_v(int row, int cg) {
  const int h = (row & 3) ^ ((row >> 2) & 1) ^ ((row >> 3) & 1);
  return cg ^ ((2 * h) & (CPR - 1));
}

// Feature held in row x of S row block rb.  Rows 4 gg + jj of blocks 2 kf and
// 2 kf + 1 hold features 32 kf + 8 gg + jj and 32 kf + 8 gg + 4 + jj, so that the
// accumulator tiles of blocks 2 kf, 2 kf + 1 are the k-fragment kf (slot e <->
// feature 32 kf + 8 g + e) of S^T as they stand.
__device__ __forceinline__ int s_feature(int rb, int x) {
  return 32 * (rb >> 1) + 8 * (x >> 2) + 4 * (rb & 1) + (x & 3);
}

// 8 consecutive elements of an LDS row stored in swizzled 16-byte chunks; `at(e)`
// is the address of element e (called with e = 0, and e = 4 for fp32).
template <typename F>
__device__ __forceinline__ void lds8(Frag<__bf16>& f, F at) {
  f.v = *reinterpret_cast<const bf16x8*>(at(0));
}
template <typename F>
__device__ __forceinline__ void lds8(Frag<float>& f, F at) {
  const float4 lo = *reinterpret_cast<const float4*>(at(0));
  const float4 hi = *reinterpret_cast<const float4*>(at(4));
  f.v[0] = lo.x; f.v[1] = lo.y; f.v[2] = lo.z; f.v[3] = lo.w;
  f.v[4] = hi.x; f.v[5] = hi.y; f.v[6] = hi.z; f.v[7] = hi.w;
}
// Store 8 fragment values to consecutive elements of a swizzled LDS row.
template <typename F>
__device__ __forceinline__ void sts8(const Frag<__bf16>& f, F at) {
  *reinterpret_cast<bf16x8*>(at(0)) = f.v;
}
template <typename F>
__device__ __forceinline__ void sts8(const Frag<float>& f, F at) {
  *reinterpret_cast<float4*>(at(0)) = float4{f.v[0], f.v[1], f.v[2], f.v[3]};
  *reinterpret_cast<float4*>(at(4)) = float4{f.v[4], f.v[5], f.v[6], f.v[7]};
}

template <typename T, int DH, int L, int MB>
__global__ __launch_bounds__(512, 1) void causal_kernel(CausalArgs a) {
  using C = CsCfg<T, DH, L, MB>;
  constexpr int KS = C::KS, FP = C::FP, NF = C::NF, RB = C::RB, VE = C::VE, CBW = C::CBW, NMW = C::NMW;
  constexpr int CPQ = FP / VE, CPK = 64 / VE, CPV = DH / VE;
  __shared__ CsLds<T, DH, L, MB> sm;

  const int head = blockIdx.x / a.parts;
  const int part = blockIdx.x - head * a.parts;
  const int hset = a.phi.per_head ? head % a.H : 0;
  pwl_load(sm.tab, a.phi.tables + (size_t)hset * kTableBytes);

  const int tid = threadIdx.x;
  const int wave = wave_id(), lane = tid % kWave;
  // lane coordinates; re-announced at the top of every chunk so that the many
  // per-lane LDS addresses derived from them are recomputed inside the loop rather
  // than hoisted out of it and kept live in registers
  int g = lane / 16, r = lane % 16;
  const int M = a.phi.M;
  const int n = a.n;
  const size_t hoff = (size_t)head * n * DH;
  const T* Q = reinterpret_cast<const T*>(a.Q) + hoff;
  const T* K = reinterpret_cast<const T*>(a.K) + hoff;
  const T* V = reinterpret_cast<const T*>(a.V) + hoff;
  T* out = reinterpret_cast<T*>(a.out) + hoff;
  const T* W = reinterpret_cast<const T*>(a.phi.W) + (size_t)hset * M * DH;
  const float* bias = a.phi.b + (size_t)hset * M;

  // chunks [0, c_begin) only build the state; chunks [c_begin, c_end) are scanned
  const int t_begin = part == 0 ? 0 : a.split;
  const int t_end = part == a.parts - 1 ? n : a.split;
  const int c_begin = t_begin / 64, c_end = (t_end + 63) / 64;

  // LDS addressing
  auto phq_at = [&](int t, int f) -> T* { return &sm.phq[t * FP + swz_rows16<CPQ>(t, f / VE) * VE + f % VE]; };
  auto phk_at = [&](int f, int t) -> T* { return &sm.phk[f * 64 + swz_k<CPK>(f, t / VE) * VE + t % VE]; };
  auto pm_at = [&](int q, int k) -> T* { return &sm.pm[q * 64 + swz_rows16<CPK>(q, k / VE) * VE + k % VE]; };
  auto vt_at = [&](int t, int c) -> T* { return &sm.vt[t * DH + swz_v<CPV>(t, c / VE) * VE + c % VE]; };

  // W fragments into LDS; P (above-diagonal blocks stay zero) and z cleared
  for (int i = tid; i < MB * KS * kWave; i += 512) {
    const int l = i % kWave, ks = (i / kWave) % KS, mb = i / (kWave * KS);
    const int p = 16 * mb + l % 16;
    Frag<T> f;
    if (p < M) load8(f, W + (size_t)p * DH + 32 * ks + 8 * (l / 16));
    else f.zero();
    store8(&sm.wfr[mb][ks][l][0], f);
  }
  for (int i = tid; i < 64 * 64; i += 512) sm.pm[i] = (T)0.0f;
  for (int i = tid; i < 2 * FP; i += 512) (&sm.zs[0][0])[i] = 0.0f;
  for (int i = tid; i < 16 * MB; i += 512) sm.bias[i] = i < M ? bias[i] : 0.0f;
  Frag<T> ones;
  ones.fill(1.0f);

  if (wave >= 4) {
    // ============================================================== map waves
    const int pw = wave - 4;  // query and key rows 16 pw .. 16 pw + 15 of every chunk
    const int mtid = tid - 256;
    Frag<T> xq[KS], xk[KS];  // query and key rows of the next chunk to map
    i32x4 vr[C::VPT];        // V of the next chunk
    auto load_rows = [&](Frag<T> (&xf)[KS], const T* X, int cc, bool live) {
      const int t = 64 * cc + 16 * pw + r;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if (live && cc < c_end && t < n) load8(xf[ks], X + (size_t)t * DH + 32 * ks + 8 * g);
        else xf[ks].zero();
      }
    };
    auto load_v = [&](i32x4 (&vf)[C::VPT], int cc) {
#pragma unroll
      for (int q = 0; q < C::VPT; ++q) {
        const int cidx = mtid + 256 * q;
        const int tt = cidx / CPV, cg = cidx % CPV;
        const int t = 64 * cc + tt;
        if (cc < c_end && t < n) vf[q] = *reinterpret_cast<const i32x4*>(V + (size_t)t * DH + cg * VE);
        else vf[q] = i32x4{0, 0, 0, 0};
      }
    };
    auto store_v = [&](const i32x4 (&vf)[C::VPT]) {
#pragma unroll
      for (int q = 0; q < C::VPT; ++q) {
        const int cidx = mtid + 256 * q;
        const int tt = cidx / CPV, cg = cidx % CPV;
        *reinterpret_cast<i32x4*>(&sm.vt[tt * DH + swz_v<CPV>(tt, cg) * VE]) = vf[q];
      }
    };
    // u for the 16 rows: query rows as u^T = W X^T (lane: projections 16 mb + 4 g + j
    // of token r), key rows as u = X W^T (lane: projection 16 mb + r of tokens 4 g + j)
    Frag<T> wreg[MB][KS];  // W fragments, loaded once (after the first barrier)
    auto project = [&](const Frag<T> (&xf)[KS], bool isq, float (&uu)[4 * MB]) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        f32x4 acc = zero4();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          if (isq) mma(acc, wreg[mb][ks], xf[ks]);
          else mma(acc, xf[ks], wreg[mb][ks]);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) uu[4 * mb + j] = acc[j] + sm.bias[16 * mb + (isq ? 4 * g + j : r)];
      }
    };
    Frag<T> qreg[C::NPQ], kreg[C::NPK];
    // z over this wave's key rows: tile mb has rows = projections 16 mb + 4 g + jj and
    // column l = channel l, accumulated from phi(K) fragments times one-hot columns
    f32x4 zacc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) zacc[mb] = zero4();
    auto add_z = [&]() {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int q = 0; q < L / 2; ++q) {
          Frag<T> oh;  // slot e holds channel 2q + (e >= 4)
          const float lo = r == 2 * q ? 1.0f : 0.0f, hi = r == 2 * q + 1 ? 1.0f : 0.0f;
          oh.set2(0, lo, lo);
          oh.set2(2, lo, lo);
          oh.set2(4, hi, hi);
          oh.set2(6, hi, hi);
          mma(zacc[mb], kreg[mb * (L / 2) + q], oh);
        }
    };
    auto write_z = [&]() {
      if (r < L) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) sm.zp[pw][(16 * mb + 4 * g + jj) * L + r] = zacc[mb][jj];
      }
    };
    // the four parts summed in a fixed order, this wave's quarter of the features
    auto sum_z = [&](int slot) {
      for (int f = FP / 4 * pw + lane; f < FP / 4 * (pw + 1); f += kWave)
        sm.zs[slot][f] = ((sm.zp[0][f] + sm.zp[1][f]) + sm.zp[2][f]) + sm.zp[3][f];
    };
    // phi(Q) of chunk cc into qreg: value (mb, j, l) at index (4 mb + j) L + l
    auto map_q = [&](const Frag<T> (&xf)[KS], int steps, int zseg, float floor) {
      float uu[4 * MB];
      project(xf, true, uu);
      int sg[4 * MB];
      pwl_search(sm.tab, steps, uu, sg);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        // one projection block (four values) at a time, so that the table reads of
        // all blocks are not hoisted together
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float y[L];
          pwl_channels<L>(sm.tab, 16 * mb + 4 * g + j < M ? sg[4 * mb + j] : zseg, floor, uu[4 * mb + j], y);
#pragma unroll
          for (int l = 0; l < L; l += 2) {
            const int idx = (4 * mb + j) * L + l;
            qreg[idx / 8].set2(idx % 8, y[l], y[l + 1]);
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    };
    auto write_q = [&]() {
      const int t = 16 * pw + r;
      if constexpr (L % 8 == 0) {
#pragma unroll
        for (int p = 0; p < C::NPQ; ++p) {
          const int mj = p / (L / 8), h = p % (L / 8);
          const int f0 = (16 * (mj / 4) + 4 * g + mj % 4) * L + 8 * h;
          sts8(qreg[p], [&](int e) { return phq_at(t, f0 + e); });
        }
      } else {
#pragma unroll
        for (int idx = 0; idx < MB * 4 * L; ++idx) {
          const int mj = idx / L, l = idx % L;
          *phq_at(t, (16 * (mj / 4) + 4 * g + mj % 4) * L + l) = (T)qreg[idx / 8].get(idx % 8);
        }
      }
    };
    // phi(K) of chunk cc into kreg: fragment (mb, q) holds channel 2q in slots 0-3 and
    // channel 2q + 1 in slots 4-7, tokens 4 g + 0..3
    auto map_k = [&](const Frag<T> (&xf)[KS], int cc, int steps, int zseg, float floor) {
      float uu[4 * MB];
      project(xf, false, uu);
      int sg[4 * MB];
      pwl_search(sm.tab, steps, uu, sg);
      const int t0 = 64 * cc + 16 * pw + 4 * g;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        __builtin_amdgcn_sched_barrier(0);
        int seg[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)  // padded projections and key rows past n give 0
          seg[j] = (16 * mb + r < M && t0 + j < n) ? sg[4 * mb + j] : zseg;
#pragma unroll
        for (int q = 0; q < L / 2; ++q) {
          float y0[4], y1[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) pwl_pair<L>(sm.tab, seg[j], q, floor, uu[4 * mb + j], y0[j], y1[j]);
          Frag<T>& f = kreg[mb * (L / 2) + q];
          f.set2(0, y0[0], y0[1]);
          f.set2(2, y0[2], y0[3]);
          f.set2(4, y1[0], y1[1]);
          f.set2(6, y1[2], y1[3]);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    };
    // Lanes g and g ^ 1 (16 apart) trade halves so that an even-g lane holds channel
    // 2q of tokens 4g .. 4g + 7 and an odd-g lane channel 2q + 1 of tokens
    // 4(g - 1) .. 4(g - 1) + 7: one 16-byte write each instead of two 8-byte ones.
    auto write_k = [&]() {
      const bool ev = (g & 1) == 0;
      const int t0 = 16 * pw + 4 * (g & ~1);
#pragma unroll
      for (int p = 0; p < C::NPK; ++p) {
        const int mb = p / (L / 2), q = p % (L / 2);
        const int f = (16 * mb + r) * L + 2 * q + (ev ? 0 : 1);
        const Frag<T>& src = kreg[p];
        if constexpr (sizeof(T) == 2) {
          typedef __attribute__((ext_vector_type(4))) int i32x4_t;
          const i32x4_t w = __builtin_bit_cast(i32x4_t, src.v);
          const int s0 = ev ? w[2] : w[0], s1 = ev ? w[3] : w[1];
          // v_permlane16_swap of a value with itself hands every lane the value of
          // lane l ^ 16: even 16-lane rows find it in the second result, odd rows in
          // the first
          const auto p0 = __builtin_amdgcn_permlane16_swap((unsigned)s0, (unsigned)s0, false, false);
          const auto p1 = __builtin_amdgcn_permlane16_swap((unsigned)s1, (unsigned)s1, false, false);
          const int r0 = (int)(ev ? p0[1] : p0[0]), r1 = (int)(ev ? p1[1] : p1[0]);
          const i32x4_t o = ev ? i32x4_t{w[0], w[1], r0, r1} : i32x4_t{r0, r1, w[2], w[3]};
          *reinterpret_cast<i32x4_t*>(phk_at(f, t0)) = o;
        } else {
          const float s0 = ev ? src.v[4] : src.v[0], s1 = ev ? src.v[5] : src.v[1];
          const float s2 = ev ? src.v[6] : src.v[2], s3 = ev ? src.v[7] : src.v[3];
          const float r0 = __shfl_xor(s0, 16, 64), r1 = __shfl_xor(s1, 16, 64);
          const float r2 = __shfl_xor(s2, 16, 64), r3 = __shfl_xor(s3, 16, 64);
          Frag<float> o;
          if (ev) {
            o.v[0] = src.v[0]; o.v[1] = src.v[1]; o.v[2] = src.v[2]; o.v[3] = src.v[3];
            o.v[4] = r0; o.v[5] = r1; o.v[6] = r2; o.v[7] = r3;
          } else {
            o.v[0] = r0; o.v[1] = r1; o.v[2] = r2; o.v[3] = r3;
            o.v[4] = src.v[4]; o.v[5] = src.v[5]; o.v[6] = src.v[6]; o.v[7] = src.v[7];
          }
          sts8(o, [&](int e) { return phk_at(f, t0 + e); });
        }
      }
    };
    // query rows are needed from chunk c_begin on, key rows and V from chunk 0
    load_rows(xq, Q, 0, 0 >= c_begin);
    load_rows(xk, K, 0, true);
    load_v(vr, 0);
    __syncthreads();  // tables, W fragments, cleared P and z
    const int steps = __builtin_amdgcn_readfirstlane(sm.tab.steps);
    const int zseg = sm.tab.zero_seg;
    const float tfloor = sm.tab.floor;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) load8(wreg[mb][ks], &sm.wfr[mb][ks][lane][0]);
    if (0 >= c_begin) {
      map_q(xq, steps, zseg, tfloor);
      write_q();
    }
    load_rows(xq, Q, 1, 1 >= c_begin);
    map_k(xk, 0, steps, zseg, tfloor);
    write_k();
    add_z();
    load_rows(xk, K, 1, true);
    store_v(vr);
    load_v(vr, 1);

    // iteration c maps chunk c + 1 (rows fetched one chunk ahead)
    for (int c = 0; c < c_end; ++c) {
      const int cn = c + 1;
      asm volatile("" : "+v"(g), "+v"(r));
      __syncthreads();  // B1
      const bool qn = cn < c_end && cn >= c_begin;
      if (qn) map_q(xq, steps, zseg, tfloor);
      load_rows(xq, Q, cn + 1, cn + 1 >= c_begin);  // also during the state-only chunks
      __syncthreads();  // B2
      if (qn) write_q();
      write_z();  // z_c, before chunk c + 1 is added
      if (cn < c_end) {
        map_k(xk, cn, steps, zseg, tfloor);
        load_rows(xk, K, cn + 1, true);
        add_z();
      }
      __syncthreads();  // B3
      sum_z(c & 1);
      if (cn < c_end) {
        write_k();
        store_v(vr);
        load_v(vr, cn + 1);
      }
    }
  } else {
    // =========================================================== matrix waves
    const int mw = wave;
    const bool active = mw < NMW;
    f32x4 sacc[CBW][RB];
#pragma unroll
    for (int x = 0; x < CBW; ++x)
#pragma unroll
      for (int i = 0; i < RB; ++i) sacc[x][i] = zero4();
    // query blocks dbase + NMW s get their phi(Q) z from this wave
    const int dbase = (mw + NMW - 2 % NMW) % NMW;
    __syncthreads();  // tables, W fragments, cleared P and z

    for (int c = 0; c < c_end; ++c) {
      const bool scan = c >= c_begin;
      const int tc = 64 * c;
      asm volatile("" : "+v"(g), "+v"(r));
      __syncthreads();  // B1: phi(Q_c), phi(K_c), V_c and z_{c-1} are in LDS
      f32x4 num[CBW][4];
      if (scan && active) {
        // P^T blocks (query block i >= key block j): rows = key tokens 16 j + 4 g + jj,
        // column = query token 16 i + r.  Each wave takes runs of blocks that share
        // their key block, so that phi(K_j) is read once per run.
        auto p_run = [&](int j, int i0, int i1) {
          Frag<T> kfr[NF];
#pragma unroll
          for (int kf = 0; kf < NF; ++kf) {
            load_tr4_at(kfr[kf], 0, lane, [&](int kk, int col) { return phk_at(32 * kf + 8 * g + kk, 16 * j + col); });
            load_tr4_at(kfr[kf], 4, lane,
                        [&](int kk, int col) { return phk_at(32 * kf + 8 * g + 4 + kk, 16 * j + col); });
          }
          for (int i = i0; i < i1; ++i) {
            f32x4 pacc = zero4();
#pragma unroll
            for (int kf = 0; kf < NF; ++kf) {
              Frag<T> qb;
              lds8(qb, [&](int e) { return phq_at(16 * i + r, 32 * kf + 8 * g + e); });
              mma(pacc, kfr[kf], qb);
            }
            if (i == j) {
#pragma unroll
              for (int jj = 0; jj < 4; ++jj)
                if (4 * g + jj > r) pacc[jj] = 0.0f;
            }
            store4(pm_at(16 * i + r, 16 * j + 4 * g), pacc[0], pacc[1], pacc[2], pacc[3]);
            float rs = (pacc[0] + pacc[1]) + (pacc[2] + pacc[3]);
            rs += __shfl_xor(rs, 16, 64);
            rs += __shfl_xor(rs, 32, 64);
            if (g == 0) sm.denp[j][16 * i + r] = rs;
          }
        };
        if constexpr (NMW == 4) {
          if (mw == 0) p_run(0, 0, 3);
          else if (mw == 1) { p_run(0, 3, 4); p_run(3, 3, 4); }
          else if (mw == 2) p_run(1, 1, 4);
          else p_run(2, 2, 4);
        } else {
          if (mw == 0) { p_run(0, 0, 4); p_run(2, 2, 4); }
          else { p_run(1, 1, 4); p_run(3, 3, 4); }
        }
        // phi(Q_c) z_{c-1} for this wave's query blocks
        const float* zprev = sm.zs[(c + 1) & 1];  // z_{c-1}
        f32x4 dacc[C::NDEN];
#pragma unroll
        for (int s = 0; s < C::NDEN; ++s) dacc[s] = zero4();
#pragma unroll
        for (int kf = 0; kf < NF; ++kf) {
          Frag<T> za;
          const float4 z0 = *reinterpret_cast<const float4*>(&zprev[32 * kf + 8 * g]);
          const float4 z1 = *reinterpret_cast<const float4*>(&zprev[32 * kf + 8 * g + 4]);
          za.set2(0, z0.x, z0.y);
          za.set2(2, z0.z, z0.w);
          za.set2(4, z1.x, z1.y);
          za.set2(6, z1.z, z1.w);
#pragma unroll
          for (int s = 0; s < C::NDEN; ++s) {
            const int i = dbase + NMW * s;
            Frag<T> qb;
            lds8(qb, [&](int e) { return phq_at(16 * i + r, 32 * kf + 8 * g + e); });
            mma(dacc[s], za, qb);
          }
        }
#pragma unroll
        for (int s = 0; s < C::NDEN; ++s)
          if (g == 0) sm.deni[16 * (dbase + NMW * s) + r] = dacc[s][0];
        // num^T = S_{c-1}^T phi(Q_c)^T
#pragma unroll
        for (int x = 0; x < CBW; ++x)
#pragma unroll
          for (int i = 0; i < 4; ++i) num[x][i] = zero4();
        // phi(Q) fragments of step kf + 1 are read while step kf multiplies
        Frag<T> qbuf[2][4];
        auto q_read = [&](Frag<T> (&qs)[4], int kf) {
#pragma unroll
          for (int i = 0; i < 4; ++i) lds8(qs[i], [&](int e) { return phq_at(16 * i + r, 32 * kf + 8 * g + e); });
        };
        q_read(qbuf[0], 0);
#pragma unroll
        for (int kf = 0; kf < NF; ++kf) {
          if (kf + 1 < NF) q_read(qbuf[(kf + 1) & 1], kf + 1);
          Frag<T> sa[CBW];
#pragma unroll
          for (int x = 0; x < CBW; ++x) {
            sa[x].set2(0, sacc[x][2 * kf][0], sacc[x][2 * kf][1]);
            sa[x].set2(2, sacc[x][2 * kf][2], sacc[x][2 * kf][3]);
            sa[x].set2(4, sacc[x][2 * kf + 1][0], sacc[x][2 * kf + 1][1]);
            sa[x].set2(6, sacc[x][2 * kf + 1][2], sacc[x][2 * kf + 1][3]);
          }
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int x = 0; x < CBW; ++x) mma(num[x][i], sa[x], qbuf[kf & 1][i]);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      __syncthreads();  // B2: P and the den parts are in LDS
      if (active) {
        Frag<T> vf[CBW][2];  // V columns 16 cb + r, tokens 32 ks + 8 g + e
#pragma unroll
        for (int x = 0; x < CBW; ++x)
#pragma unroll
          for (int ks = 0; ks < 2; ++ks) {
            const int c0 = 16 * (CBW * mw + x);
            load_tr4_at(vf[x][ks], 0, lane, [&](int kk, int col) { return vt_at(32 * ks + 8 * g + kk, c0 + col); });
            load_tr4_at(vf[x][ks], 4, lane,
                        [&](int kk, int col) { return vt_at(32 * ks + 8 * g + 4 + kk, c0 + col); });
          }
        if (scan) {
          // num^T += V^T P^T over the key tokens at or before each query block
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int ks = 0; ks < 2; ++ks)
              if (2 * ks <= i) {
                Frag<T> pb;
                lds8(pb, [&](int e) { return pm_at(16 * i + r, 32 * ks + 8 * g + e); });
#pragma unroll
                for (int x = 0; x < CBW; ++x) mma(num[x][i], vf[x][ks], pb);
              }
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int q = 16 * i + r;
            float den = sm.deni[q];
#pragma unroll
            for (int j = 0; j <= i; ++j) den += sm.denp[j][q];
            const int t = tc + q;
            if (t < t_end) {
              const float rinv = 1.0f / (den + ldexpf(a.eps, 2 * sm.tab.scale_exp));
#pragma unroll
              for (int x = 0; x < CBW; ++x)
                store4(out + (size_t)t * DH + 16 * (CBW * mw + x) + 4 * g, num[x][i][0] * rinv,
                       num[x][i][1] * rinv, num[x][i][2] * rinv, num[x][i][3] * rinv);
            }
          }
        }
        // S += phi(K_c)^T V_c (rows in s_feature order)
        // fragments read kPre ahead of their use
        constexpr int kPre = 4;
        auto ka_read = [&](Frag<T>& f, int idx) {
          const int rb = idx / 2, ks = idx % 2;
          lds8(f, [&](int e) { return phk_at(s_feature(rb, r), 32 * ks + 8 * g + e); });
        };
        Frag<T> kb[kPre];
#pragma unroll
        for (int p = 0; p < kPre; ++p) ka_read(kb[p], p);
#pragma unroll
        for (int idx = 0; idx < 2 * RB; ++idx) {
          const Frag<T> ka = kb[idx % kPre];
          if (idx + kPre < 2 * RB) ka_read(kb[idx % kPre], idx + kPre);
#pragma unroll
          for (int x = 0; x < CBW; ++x) mma(sacc[x][idx / 2], ka, vf[x][idx % 2]);
        }
      }
      __syncthreads();  // B3: phi(K_c) and V_c are no longer read
    }
  }
}

template <typename T, int DH, int L, int MB>
static hipError_t cs_run(const CausalArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((causal_kernel<T, DH, L, MB>), dim3(a.heads * a.parts), dim3(512), 0, s, a);
  return hipGetLastError();
}

// (dtype, d, L, projection blocks) combinations that are built.
#define LUNA_CS_CASES(X) \
  X(float, 32, 8, 1)     \
  X(float, 32, 2, 1)     \
  X(float, 64, 8, 1)     \
  X(__bf16, 32, 8, 1)    \
  X(__bf16, 64, 8, 1)    \
  X(__bf16, 64, 8, 2)    \
  X(__bf16, 128, 8, 1)   \
  X(__bf16, 128, 8, 2)

template <typename T>
static constexpr Dt cs_dt_of() { return sizeof(T) == 2 ? Dt::BF16 : Dt::F32; }

bool causal_supported(Dt dt, int d, int L, int M) {
  const int MB = (M + 15) / 16;
#define X(T_, D_, L_, MB_) \
  if (dt == cs_dt_of<T_>() && d == D_ && L == L_ && MB == MB_) return true;
  LUNA_CS_CASES(X)
#undef X
  return false;
}

hipError_t launch_causal(Dt dt, int d, int L, int M, const CausalArgs& a, hipStream_t s) {
  const int MB = (M + 15) / 16;
#define X(T_, D_, L_, MB_) \
  if (dt == cs_dt_of<T_>() && d == D_ && L == L_ && MB == MB_) return cs_run<T_, D_, L_, MB_>(a, s);
  LUNA_CS_CASES(X)
#undef X
  return hipErrorInvalidValue;
}

}  // namespace luna
