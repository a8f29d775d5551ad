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
// Waves.  Wave w owns value columns 16w .. 16w + 15 (d / 16 waves) and keeps the
// matching slice of S (all features) in fp32 matrix-core accumulators.  Per chunk,
// with phi(Q_c), phi(K_c) and V_c already in LDS:
//   - its share of the P^T blocks (P and its row sums to LDS) and of
//     phi(Q_c) z_{c-1} (to LDS);
//   - num^T = S_{c-1}^T phi(Q_c)^T for its columns, with S taken straight from the
//     accumulators: the feature order of S's rows is chosen so that two
//     accumulator tiles form one k-fragment of S^T;
//   - S += phi(K_c)^T V_c and z += phi(K_c)^T 1;
//   - barrier; num^T += V^T P^T; divide; store;
//   - phi of its 16-row blocks of chunk c + 1 (query rows or key rows) and its
//     share of V_{c+1} into LDS.
// Two barriers per chunk.  phi(Q) is kept token-major and phi(K) feature-major in
// LDS, so every large operand is one 16-byte read per lane; only the P^T blocks
// (phi(K) rows) and V use the gfx950 transpose read.  Every LDS tile is stored in
// 16-byte chunks XOR-swizzled by row so that the rows one read touches fall in
// distinct banks.
#include "luna_device.hpp"
#include "luna_kernels.hpp"

namespace luna {

template <typename T, int DH, int L, int MB>
struct CsCfg {
  static constexpr int NW = DH / 16;              // waves, one 16-column block of values each
  static constexpr int NT = NW * kWave;
  static constexpr int KS = DH / 32;              // 32-wide k-steps of the projection
  static constexpr int FP = 16 * MB * L;          // features, projections padded to 16
  static constexpr int NF = FP / 32;              // 32-feature k-fragments
  static constexpr int RB = FP / 16;              // 16-feature row blocks of S
  static constexpr int RBZ = (RB + NW - 1) / NW;  // row blocks of z per wave
  static constexpr int VE = 16 / (int)sizeof(T);  // elements per 16-byte chunk
  static constexpr int NTASK = 8 / NW;            // 16-row phi blocks per wave per chunk (4 Q + 4 K)
  static constexpr int VPT = 64 * DH / VE / NT;   // 16-byte V chunks per thread
  static constexpr int NDEN = NW >= 4 ? 1 : 4 / NW;  // query blocks whose phi(Q) z a wave forms
  static constexpr int NSEG = nseg_cap(L, kAttnSegBytes);
  static_assert(NW >= 2 && 8 % NW == 0, "d must be 32, 64 or 128");
  static_assert(FP % 32 == 0 && L % 2 == 0, "features must fill 32-wide fragments");
};

template <typename T, int DH, int L, int MB>
struct CsLds {
  using C = CsCfg<T, DH, L, MB>;
  PwlLds<L, C::NSEG> tab;
  alignas(16) T wfr[MB][C::KS][kWave][8];  // W fragments (A of u^T = W X^T, B of u = X W^T)
  alignas(16) T phq[64 * C::FP];           // phi(Q_c), token-major
  alignas(16) T phk[C::FP * 64];           // phi(K_c)^T, feature-major
  alignas(16) T pm[64 * 64];               // P, query-major (blocks above the diagonal stay 0)
  alignas(16) T vt[64 * DH];               // V_c, token-major
  alignas(16) float denp[4][64];           // row sums of P per key block
  alignas(16) float deni[64];              // phi(Q_c) z_{c-1}
  alignas(16) float zb[2][C::FP];          // z by chunk parity
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
// bits 0, 1, 3 and 4.
template <int CPR>
__device__ __forceinline__ int swz_k(int row, int cg) {
  if constexpr (CPR >= 16) return cg ^ ((row & 3) | ((row >> 1) & 12));
  else return cg ^ (((row >> 1) & 1) | ((row >> 2) & 6));
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
__global__ __launch_bounds__(64 * (DH / 16), 1) void causal_kernel(CausalArgs a) {
  using C = CsCfg<T, DH, L, MB>;
  constexpr int NW = C::NW, KS = C::KS, FP = C::FP, NF = C::NF, RB = C::RB, VE = C::VE;
  constexpr int CPQ = FP / VE, CPK = 64 / VE, CPV = DH / VE;
  __shared__ CsLds<T, DH, L, MB> sm;

  const int head = blockIdx.x / a.parts;
  const int part = blockIdx.x - head * a.parts;
  const int hset = a.phi.per_head ? head % a.H : 0;
  pwl_load(sm.tab, a.phi.tables + (size_t)hset * kTableBytes);

  const int tid = threadIdx.x;
  const int wave = wave_id(), lane = tid % kWave;
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
  for (int i = tid; i < MB * KS * kWave; i += C::NT) {
    const int l = i % kWave, ks = (i / kWave) % KS, mb = i / (kWave * KS);
    const int p = 16 * mb + l % 16;
    Frag<T> f;
    if (p < M) load8(f, W + (size_t)p * DH + 32 * ks + 8 * (l / 16));
    else f.zero();
    store8(&sm.wfr[mb][ks][l][0], f);
  }
  for (int i = tid; i < 64 * 64; i += C::NT) sm.pm[i] = (T)0.0f;
  for (int i = tid; i < 2 * FP; i += C::NT) (&sm.zb[0][0])[i] = 0.0f;

  // projection biases: rows 16 mb + 4 g + j (u^T layout) and column 16 mb + r (u layout)
  float brow[MB][4], bcol[MB];
  bool prow[MB][4], pcol[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    pcol[mb] = 16 * mb + r < M;
    bcol[mb] = pcol[mb] ? bias[16 * mb + r] : 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = 16 * mb + 4 * g + j;
      prow[mb][j] = i < M;
      brow[mb][j] = i < M ? bias[i] : 0.0f;
    }
  }
  Frag<T> ones;
  ones.fill(1.0f);

  // ---- phi blocks of this wave: task k is block b = wave + NW k (0-3: Q, 4-7: K) ----
  auto task_q = [&](int k) { return wave + NW * k < 4; };
  auto task_blk = [&](int k) { return (wave + NW * k) & 3; };
  // does task k map chunk cc (key blocks always, query blocks only where scanned)
  auto task_live = [&](int k, int cc) { return cc < c_end && (!task_q(k) || cc >= c_begin); };

  Frag<T> xf[C::NTASK][KS];  // X rows of the next chunk to map
  auto load_x = [&](int k, int cc) {
    const T* X = task_q(k) ? Q : K;
    const int t = 64 * cc + 16 * task_blk(k) + r;
    const bool live = task_live(k, cc) && t < n;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (live) load8(xf[k][ks], X + (size_t)t * DH + 32 * ks + 8 * g);
      else xf[k][ks].zero();
    }
  };

  // phi of block task k of chunk cc, written to LDS.  Query rows: u^T = W X^T, the
  // lane holds projections 16 mb + 4 g + j of token r and writes features
  // (16 mb + 4 g + j) L + l of that token.  Key rows: u = X W^T, the lane holds
  // projection 16 mb + r of tokens 4 g + j and writes, for each channel l, the four
  // tokens of feature (16 mb + r) L + l.
  auto map_block = [&](int k, int cc, int steps, int zseg, float floor) {
    float uu[4 * MB];
    const bool isq = task_q(k);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      f32x4 acc = zero4();
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        Frag<T> wf;
        load8(wf, &sm.wfr[mb][ks][lane][0]);
        if (isq) mma(acc, wf, xf[k][ks]);
        else mma(acc, xf[k][ks], wf);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) uu[4 * mb + j] = acc[j] + (isq ? brow[mb][j] : bcol[mb]);
    }
    int sg[4 * MB];
    pwl_search(sm.tab, steps, uu, sg);
    const int blk = task_blk(k);
    if (isq) {
      const int t = 16 * blk + r;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int seg = prow[mb][j] ? sg[4 * mb + j] : zseg;  // padded projections give 0
          const int f0 = (16 * mb + 4 * g + j) * L;
          float y[L];
          pwl_channels<L>(sm.tab, seg, floor, uu[4 * mb + j], y);
          if constexpr (L % 8 == 0) {
#pragma unroll
            for (int h = 0; h < L / 8; ++h) {
              Frag<T> f;
#pragma unroll
              for (int e = 0; e < 8; e += 2) f.set2(e, y[8 * h + e], y[8 * h + e + 1]);
              sts8(f, [&](int e) { return phq_at(t, f0 + 8 * h + e); });
            }
          } else {
#pragma unroll
            for (int l = 0; l < L; ++l) *phq_at(t, f0 + l) = (T)y[l];
          }
        }
    } else {
      const int t0 = 64 * cc + 16 * blk + 4 * g;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        int seg[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)  // padded projections and key rows past n give 0
          seg[j] = (pcol[mb] && t0 + j < n) ? sg[4 * mb + j] : zseg;
#pragma unroll
        for (int q = 0; q < L / 2; ++q) {
          float y0[4], y1[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) pwl_pair<L>(sm.tab, seg[j], q, floor, uu[4 * mb + j], y0[j], y1[j]);
          const int f = (16 * mb + r) * L + 2 * q;
          store4(phk_at(f, 16 * blk + 4 * g), y0[0], y0[1], y0[2], y0[3]);
          store4(phk_at(f + 1, 16 * blk + 4 * g), y1[0], y1[1], y1[2], y1[3]);
        }
      }
    }
  };
  // V tile of chunk cc through registers
  i32x4 vpf[C::VPT];
  auto load_v = [&](int cc) {
#pragma unroll
    for (int q = 0; q < C::VPT; ++q) {
      const int cidx = tid + C::NT * q;
      const int tt = cidx / CPV, cg = cidx % CPV;
      const int t = 64 * cc + tt;
      if (t < n && cc < c_end) vpf[q] = *reinterpret_cast<const i32x4*>(V + (size_t)t * DH + cg * VE);
      else vpf[q] = i32x4{0, 0, 0, 0};
    }
  };
  auto commit_v = [&]() {
#pragma unroll
    for (int q = 0; q < C::VPT; ++q) {
      const int cidx = tid + C::NT * q;
      const int tt = cidx / CPV, cg = cidx % CPV;
      *reinterpret_cast<i32x4*>(&sm.vt[tt * DH + swz_v<CPV>(tt, cg) * VE]) = vpf[q];
    }
  };

  // ---- prologue: chunk 0 into LDS ----
#pragma unroll
  for (int k = 0; k < C::NTASK; ++k) load_x(k, 0);
  load_v(0);
  __syncthreads();  // tables, W fragments, cleared P and z
  const int steps = __builtin_amdgcn_readfirstlane(sm.tab.steps);
  const int zseg = sm.tab.zero_seg;
  const float tfloor = sm.tab.floor;
#pragma unroll
  for (int k = 0; k < C::NTASK; ++k)
    if (task_live(k, 0)) map_block(k, 0, steps, zseg, tfloor);
  commit_v();
#pragma unroll
  for (int k = 0; k < C::NTASK; ++k) load_x(k, 1);
  load_v(1);

  f32x4 sacc[RB];
  f32x4 zacc[C::RBZ];
#pragma unroll
  for (int i = 0; i < RB; ++i) sacc[i] = zero4();
#pragma unroll
  for (int i = 0; i < C::RBZ; ++i) zacc[i] = zero4();
  // query blocks dbase, dbase + NW, ... (below 4) get their phi(Q) z from this wave
  const int dbase = (wave + NW - 2 % NW) % NW;

  for (int c = 0; c < c_end; ++c) {
    const bool scan = c >= c_begin;
    const int tc = 64 * c;
    __syncthreads();  // chunk c's phi and V, and z_{c-1}, are in LDS

    f32x4 num[4];
    if (scan) {
      // P^T blocks (query block i >= key block j), enumerated key block by key
      // block: rows = key tokens 16 j + 4 g + jj, column = query token 16 i + r
      for (int task = wave; task < 10; task += NW) {
        const int j = task < 4 ? 0 : (task < 7 ? 1 : (task < 9 ? 2 : 3));
        const int i = task - (j == 0 ? 0 : (j == 1 ? 4 : (j == 2 ? 7 : 9))) + j;
        f32x4 pacc = zero4();
#pragma unroll
        for (int kf = 0; kf < NF; ++kf) {
          Frag<T> ka, qb;
          load_tr4_at(ka, 0, lane, [&](int kk, int col) { return phk_at(32 * kf + 8 * g + kk, 16 * j + col); });
          load_tr4_at(ka, 4, lane, [&](int kk, int col) { return phk_at(32 * kf + 8 * g + 4 + kk, 16 * j + col); });
          lds8(qb, [&](int e) { return phq_at(16 * i + r, 32 * kf + 8 * g + e); });
          mma(pacc, ka, qb);
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
      // num^T = S_{c-1}^T phi(Q_c)^T; phi(Q_c) z_{c-1} for this wave's query blocks
      f32x4 dacc[C::NDEN];
#pragma unroll
      for (int s = 0; s < C::NDEN; ++s) dacc[s] = zero4();
#pragma unroll
      for (int i = 0; i < 4; ++i) num[i] = zero4();
      const float* zprev = sm.zb[(c + 1) & 1];
#pragma unroll
      for (int kf = 0; kf < NF; ++kf) {
        Frag<T> sa;
        sa.set2(0, sacc[2 * kf][0], sacc[2 * kf][1]);
        sa.set2(2, sacc[2 * kf][2], sacc[2 * kf][3]);
        sa.set2(4, sacc[2 * kf + 1][0], sacc[2 * kf + 1][1]);
        sa.set2(6, sacc[2 * kf + 1][2], sacc[2 * kf + 1][3]);
        Frag<T> za;
        if (dbase < 4) {
          const float4 z0 = *reinterpret_cast<const float4*>(&zprev[32 * kf + 8 * g]);
          const float4 z1 = *reinterpret_cast<const float4*>(&zprev[32 * kf + 8 * g + 4]);
          za.set2(0, z0.x, z0.y);
          za.set2(2, z0.z, z0.w);
          za.set2(4, z1.x, z1.y);
          za.set2(6, z1.z, z1.w);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          Frag<T> qb;
          lds8(qb, [&](int e) { return phq_at(16 * i + r, 32 * kf + 8 * g + e); });
          mma(num[i], sa, qb);
#pragma unroll
          for (int s = 0; s < C::NDEN; ++s)
            if (dbase + NW * s == i) mma(dacc[s], za, qb);
        }
      }
#pragma unroll
      for (int s = 0; s < C::NDEN; ++s)
        if (dbase + NW * s < 4 && g == 0) sm.deni[16 * (dbase + NW * s) + r] = dacc[s][0];
    }

    // S += phi(K_c)^T V_c (rows in s_feature order), z alongside
    Frag<T> vf[2];  // V columns 16 w + r, tokens 32 ks + 8 g + e
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      load_tr4_at(vf[ks], 0, lane, [&](int kk, int col) { return vt_at(32 * ks + 8 * g + kk, 16 * wave + col); });
      load_tr4_at(vf[ks], 4, lane, [&](int kk, int col) { return vt_at(32 * ks + 8 * g + 4 + kk, 16 * wave + col); });
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int frow = s_feature(rb, r);
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        Frag<T> ka;
        lds8(ka, [&](int e) { return phk_at(frow, 32 * ks + 8 * g + e); });
        mma(sacc[rb], ka, vf[ks]);
        if (rb % NW == wave) mma(zacc[rb / NW], ka, ones);
      }
    }
    // z_c to LDS: column 0 of the z tiles, rows 4 g + jj = features s_feature(rb, 4 g + jj)
#pragma unroll
    for (int i = 0; i < C::RBZ; ++i) {
      const int rb = wave + NW * i;
      if (rb < RB && r == 0)
        *reinterpret_cast<float4*>(&sm.zb[c & 1][s_feature(rb, 4 * g)]) =
            float4{zacc[i][0], zacc[i][1], zacc[i][2], zacc[i][3]};
    }

    __syncthreads();  // phi(Q_c), phi(K_c) and V_c are no longer read; P and the den parts are written

    if (scan) {
      // num^T += V^T P^T over the key tokens at or before each query block
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
          if (2 * ks <= i) {
            Frag<T> pb;
            lds8(pb, [&](int e) { return pm_at(16 * i + r, 32 * ks + 8 * g + e); });
            mma(num[i], vf[ks], pb);
          }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = 16 * i + r;
        float den = sm.deni[q];
#pragma unroll
        for (int j = 0; j <= i; ++j) den += sm.denp[j][q];
        const int t = tc + q;
        if (t < t_end) {
          const float rinv = 1.0f / (den + a.eps);
          store4(out + (size_t)t * DH + 16 * wave + 4 * g, num[i][0] * rinv, num[i][1] * rinv, num[i][2] * rinv,
                 num[i][3] * rinv);
        }
      }
    }

    // phi and V of chunk c + 1 into LDS, then fetch chunk c + 2
#pragma unroll
    for (int k = 0; k < C::NTASK; ++k)
      if (task_live(k, c + 1)) map_block(k, c + 1, steps, zseg, tfloor);
    if (c + 1 < c_end) commit_v();
#pragma unroll
    for (int k = 0; k < C::NTASK; ++k) load_x(k, c + 2);
    load_v(c + 2);
  }
}

template <typename T, int DH, int L, int MB>
static hipError_t cs_run(const CausalArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((causal_kernel<T, DH, L, MB>), dim3(a.heads * a.parts), dim3(CsCfg<T, DH, L, MB>::NT), 0, s,
                     a);
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
