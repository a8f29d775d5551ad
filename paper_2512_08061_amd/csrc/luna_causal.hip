// luna_causal.hip -- causal (streaming) LUNA attention as a chunked prefix scan.
//
// out_t = phi(q_t)^T S_t / (phi(q_t)^T z_t + eps) with S_t, z_t summed over s <= t.
// Tokens are processed in chunks of 64; within chunk c (query rows t, key columns s):
//
//   P      = tril(phi(Q_c) phi(K_c)^T)              (diagonal included)
//   num    = P V_c + phi(Q_c) S_{c-1},   den = P 1 + phi(Q_c) z_{c-1}
//   S_c    = S_{c-1} + phi(K_c)^T V_c,   z_c = z_{c-1} + phi(K_c)^T 1
//
// which regroups the prefix sums exactly.  One workgroup of 8 waves owns one
// (head, tile of DVT value columns) and walks the chunks in order, keeping S in
// fp32 matrix-core accumulators; there is no cross-workgroup traffic.
//
// The waves are specialised and software-pipelined across chunks, so that the
// vector work of the feature map (chunk c + 1) and the matrix work of the
// attention (chunk c) sit in the same straight-line region of every wave:
//
//  query waves 0-3 (token block b = w):  readout of query block b of chunk c --
//     P^T blocks j = phi(K_j) phi(Q_b)^T for all four key blocks (blocks after b and
//     the upper part of the diagonal block zeroed), num^T += V^T P^T and
//     den += 1^T P^T, then num^T += S_{c-1}^T phi(Q_b)^T, den += z_{c-1}^T phi(Q_b)^T,
//     out = num * (1 / (den + eps));  then phi(Q) of block b of chunk c + 1, kept
//     in registers for the next iteration.
//  key waves 4-7 (token block b = w - 4):  S += phi(K_c)^T V_c for S row blocks
//     4(w-4) .. 4(w-4)+3 (z alongside), then phi(K) of block b of chunk c + 1 into
//     the other half of a double-buffered LDS array; at the start of each iteration
//     they stage S_{c-1}, z_{c-1} to LDS as the query waves' A operands.
//
// phi: u^T = W X^T on the matrix cores (W fragments from LDS), one batched search
// of the piecewise-linear table, L fused multiply-adds per projection; the result
// is k-order fragments (lane = token, 8 features).  Padded projections and key
// tokens past n select the table's all-zero segment.  V^T and phi(K)^T operands
// come from row-major LDS tiles through the gfx950 transpose read.  Two workgroup
// barriers per chunk; Q/K rows are fetched two chunks ahead, V one chunk ahead.
#include "luna_device.hpp"
#include "luna_kernels.hpp"

namespace luna {

template <typename T, int DH, int L, int MB, int DVT>
struct CsCfg {
  static constexpr int KS = DH / 32;
  static constexpr int NF = (4 * MB * L + 7) / 8;   // k-order fragments over features
  static constexpr int FR = NF * 32;                // padded feature rows of S
  static constexpr int RB = FR / 16;                // row blocks of S
  static constexpr int RBK = (RB + 3) / 4;          // row blocks per key wave
  static constexpr int CBT = DVT / 16;              // column blocks of the tile
  static constexpr int NSEG = nseg_cap(L, kAttnSegBytes);
  static constexpr int VE = 16 / (int)sizeof(T);    // elements per 16-byte chunk
  static constexpr int VROW = DVT;                  // V-tile row (elements), chunks swizzled
  static constexpr int VCPR = DVT / VE;             // 16-byte chunks per V-tile row
  static constexpr int VCH = 64 * DVT / VE;         // 16-byte chunks in a V tile
  static constexpr int NVC = (VCH + 511) / 512;     // per thread
};

// Physical 16-byte chunk of logical chunk cg in V-tile row `row`: an XOR swizzle
// that spreads the four (and eight) consecutive rows read by one transposed load
// over distinct banks.
template <int CPR>
__device__ __forceinline__ int vswz(int row, int cg) {
  const int h = (row & 3) ^ ((row >> 2) & 1) ^ ((row >> 3) & 1);
  return cg ^ ((2 * h) & (CPR - 1));
}

template <typename T, int DH, int L, int MB, int DVT>
struct CsLds {
  using C = CsCfg<T, DH, L, MB, DVT>;
  PwlLds<L, C::NSEG> tab;
  alignas(16) T wfr[MB][C::KS][kWave][8];       // W as A fragments of u^T = W X^T
  alignas(16) T pk[2][4][C::NF][kWave][8];      // phi(K) fragments, by chunk parity
  alignas(16) T vtile[64][C::VROW];             // V tile, row-major (token x column)
  alignas(16) T sst[C::CBT][C::NF][kWave][8];   // S_{c-1} as A fragments
  alignas(16) T zst[C::NF][4][8];               // z_{c-1} as A fragment slots per lane group
};

template <typename T, int DH, int L, int MB, int DVT>
__global__ __launch_bounds__(512, 1) void causal_kernel(CausalArgs a) {
  using C = CsCfg<T, DH, L, MB, DVT>;
  __shared__ CsLds<T, DH, L, MB, DVT> sm;

  const int head = blockIdx.x / a.dv_tiles;
  const int c0 = (blockIdx.x - head * a.dv_tiles) * DVT;
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

  const int role = wave / 4;   // 0: queries and readout, 1: keys and state update
  const int blk = wave % 4;    // token block of the chunk this wave maps
  const T* X = role ? K : Q;

  // W fragments into LDS; S and z start at zero
  for (int i = tid; i < MB * C::KS * kWave; i += 512) {
    const int l = i % kWave, ks = (i / kWave) % C::KS, mb = i / (kWave * C::KS);
    const int p = 16 * mb + l % 16;
    Frag<T> f;
    if (p < M) load8(f, W + (size_t)p * DH + 32 * ks + 8 * (l / 16));
    else f.zero();
    store8(&sm.wfr[mb][ks][l][0], f);
  }
  for (int i = tid; i < C::CBT * C::NF * kWave; i += 512) {
    Frag<T> f;
    f.zero();
    store8(&sm.sst[0][0][0][0] + (size_t)i * 8, f);
  }
  for (int i = tid; i < C::NF * 4; i += 512) {
    Frag<T> f;
    f.zero();
    store8(&sm.zst[0][0][0] + (size_t)i * 8, f);
  }
  float brow[MB][4];
  bool pok[MB][4];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = 16 * mb + 4 * g + j;
      pok[mb][j] = i < M;
      brow[mb][j] = i < M ? bias[i] : 0.0f;
    }
  Frag<T> ones;
  ones.fill(1.0f);
  const int nchunks = (n + 63) / 64;

  // X rows of this wave's block of chunk cc (zero past n or past the last chunk)
  auto load_x = [&](Frag<T> (&xf)[C::KS], int cc) {
    const int t = 64 * cc + 16 * blk + r;
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      if (t < n) load8(xf[ks], X + (size_t)t * DH + 32 * ks + 8 * g);
      else xf[ks].zero();
    }
  };
  // this thread's share of the V tile of chunk cc
  auto load_v = [&](i32x4 (&vf)[C::NVC], int cc) {
#pragma unroll
    for (int q = 0; q < C::NVC; ++q) {
      const int cidx = tid + 512 * q;
      const int tt = cidx / (DVT / C::VE), cg = cidx % (DVT / C::VE);
      const int tv = 64 * cc + tt;
      if (cidx < C::VCH && tv < n) vf[q] = *reinterpret_cast<const i32x4*>(V + (size_t)tv * DH + c0 + cg * C::VE);
      else vf[q] = i32x4{0, 0, 0, 0};
    }
  };
  auto store_v = [&](const i32x4 (&vf)[C::NVC]) {
#pragma unroll
    for (int q = 0; q < C::NVC; ++q) {
      const int cidx = tid + 512 * q;
      if (cidx < C::VCH) {
        const int tt = cidx / (DVT / C::VE), cg = cidx % (DVT / C::VE);
        *reinterpret_cast<i32x4*>(&sm.vtile[tt][vswz<C::VCPR>(tt, cg) * C::VE]) = vf[q];
      }
    }
  };

  // element (row, col) of the swizzled V tile
  auto v_at = [&](int row, int col) -> const T* {
    return &sm.vtile[row][vswz<C::VCPR>(row, col / C::VE) * C::VE + col % C::VE];
  };

  __syncthreads();
  const int tsteps = __builtin_amdgcn_readfirstlane(sm.tab.steps);
  const int zseg = sm.tab.zero_seg;
  const float tfloor = sm.tab.floor;

  // phi of this wave's 16 rows of chunk cc
  auto feature_map = [&](const Frag<T> (&xf)[C::KS], int cc, Frag<T> (&ph)[C::NF]) {
    const bool tok_ok = 64 * cc + 16 * blk + r < n;
    float uu[4 * MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      f32x4 acc = zero4();
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) {
        Frag<T> wa;
        load8(wa, &sm.wfr[mb][ks][lane][0]);
        mma(acc, wa, xf[ks]);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) uu[4 * mb + j] = acc[j] + brow[mb][j];
    }
    int sg[4 * MB];
    pwl_search(sm.tab, tsteps, uu, sg);
    const bool kill_tok = role && !tok_ok;  // key rows past n contribute nothing
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (!pok[mb][j] || kill_tok) sg[4 * mb + j] = zseg;
#pragma unroll
    for (int k = 0; k < C::NF; ++k) ph[k].zero();
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float y[L];
        pwl_channels<L>(sm.tab, sg[4 * mb + j], tfloor, uu[4 * mb + j], y);
#pragma unroll
        for (int l = 0; l < L; ++l) {
          const int p = (mb * 4 + j) * L + l;
          if constexpr (L % 2 == 0) {
            if (l % 2 == 0) ph[p / 8].set2(p % 8, y[l], y[l + 1]);
          } else {
            ph[p / 8].set(p % 8, y[l]);
          }
        }
      }
  };

  Frag<T> xa[C::KS], xb[C::KS];  // X rows of chunks c + 1 and c + 2
  i32x4 vn[C::NVC];              // V tile of chunk c (written at the top of iteration c)
  load_x(xa, 0);
  load_x(xb, 1);
  load_v(vn, 0);

  if (role == 0) {
    // ------------------------------------------------------------ query waves
    Frag<T> pq[C::NF];
    feature_map(xa, 0, pq);
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) xa[ks] = xb[ks];
    load_x(xb, 2);
    for (int c = 0; c < nchunks; ++c) {
      const int tc = 64 * c;
      const int par = c & 1;
      __syncthreads();  // previous chunk's readers are done with the V tile and S staging
      store_v(vn);
      __syncthreads();  // V_c, S_{c-1}, z_{c-1} and phi(K_c) visible
      load_v(vn, c + 1);

      // P^T blocks against the four key blocks
      f32x4 pacc[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        pacc[j] = zero4();
#pragma unroll
        for (int k = 0; k < C::NF; ++k) {
          Frag<T> ka;
          load8(ka, &sm.pk[par][j][k][lane][0]);
          mma(pacc[j], ka, pq[k]);
        }
      }
      // keep key token 16 j + 4 g + jj <= query token 16 blk + r
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const bool keep = (j < blk) || (j == blk && 4 * g + jj <= r);
          pacc[j][jj] = keep ? pacc[j][jj] : 0.0f;
        }
      f32x4 num[C::CBT], den = zero4();
#pragma unroll
      for (int cb = 0; cb < C::CBT; ++cb) num[cb] = zero4();
#pragma unroll
      for (int pr = 0; pr < 2; ++pr) {
        const int j0 = 2 * pr, j1 = 2 * pr + 1;
        Frag<T> bp;
        bp.set2(0, pacc[j0][0], pacc[j0][1]);
        bp.set2(2, pacc[j0][2], pacc[j0][3]);
        bp.set2(4, pacc[j1][0], pacc[j1][1]);
        bp.set2(6, pacc[j1][2], pacc[j1][3]);
        mma(den, ones, bp);
#pragma unroll
        for (int cb = 0; cb < C::CBT; ++cb) {
          Frag<T> va;
          load_tr4_at(va, 0, lane, [&](int kk, int col) { return v_at(16 * j0 + 4 * g + kk, 16 * cb + col); });
          load_tr4_at(va, 4, lane, [&](int kk, int col) { return v_at(16 * j1 + 4 * g + kk, 16 * cb + col); });
          mma(num[cb], va, bp);
        }
      }
#pragma unroll
      for (int k = 0; k < C::NF; ++k) {
#pragma unroll
        for (int cb = 0; cb < C::CBT; ++cb) {
          Frag<T> sa;
          load8(sa, &sm.sst[cb][k][lane][0]);
          mma(num[cb], sa, pq[k]);
        }
        Frag<T> za;
        load8(za, &sm.zst[k][g][0]);
        mma(den, za, pq[k]);
      }
      {
        const int t = tc + 16 * blk + r;
        if (t < n) {
          const float rinv = 1.0f / (den[0] + a.eps);
          T* o = out + (size_t)t * DH + c0 + 4 * g;
#pragma unroll
          for (int cb = 0; cb < C::CBT; ++cb)
            store4(o + 16 * cb, num[cb][0] * rinv, num[cb][1] * rinv, num[cb][2] * rinv, num[cb][3] * rinv);
        }
      }
      // phi(Q) of the next chunk
      feature_map(xa, c + 1, pq);
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) xa[ks] = xb[ks];
      load_x(xb, c + 3);
    }
  } else {
    // -------------------------------------------------------------- key waves
    {
      Frag<T> ph[C::NF];
      feature_map(xa, 0, ph);
#pragma unroll
      for (int k = 0; k < C::NF; ++k) store8(&sm.pk[0][blk][k][lane][0], ph[k]);
    }
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) xa[ks] = xb[ks];
    load_x(xb, 2);
    f32x4 sacc[C::RBK][C::CBT];
    f32x4 zacc[C::RBK];
#pragma unroll
    for (int i = 0; i < C::RBK; ++i) {
      zacc[i] = zero4();
#pragma unroll
      for (int cb = 0; cb < C::CBT; ++cb) sacc[i][cb] = zero4();
    }
    for (int c = 0; c < nchunks; ++c) {
      const int par = c & 1;
      __syncthreads();  // query waves are done with the previous staging and V tile
      store_v(vn);
      // stage S_{c-1}, z_{c-1}
#pragma unroll
      for (int i = 0; i < C::RBK; ++i) {
        const int rb = C::RBK * blk + i;
        if (rb < C::RB) {
          const int k = rb / 2, gp = 2 * (rb % 2) + g / 2, e0 = 4 * (g % 2);
#pragma unroll
          for (int cb = 0; cb < C::CBT; ++cb)
            store4(&sm.sst[cb][k][16 * gp + r][e0], sacc[i][cb][0], sacc[i][cb][1], sacc[i][cb][2], sacc[i][cb][3]);
          if (r == 0) store4(&sm.zst[k][gp][e0], zacc[i][0], zacc[i][1], zacc[i][2], zacc[i][3]);
        }
      }
      __syncthreads();  // V_c and the staged state visible
      load_v(vn, c + 1);

      // S += phi(K_c)^T V_c over the chunk's 64 key tokens
#pragma unroll
      for (int ks2 = 0; ks2 < 2; ++ks2) {
        Frag<T> bv[C::CBT];
#pragma unroll
        for (int cb = 0; cb < C::CBT; ++cb) {
          load_tr4_at(bv[cb], 0, lane, [&](int kk, int col) { return v_at(32 * ks2 + 8 * g + kk, 16 * cb + col); });
          load_tr4_at(bv[cb], 4, lane, [&](int kk, int col) { return v_at(32 * ks2 + 8 * g + 4 + kk, 16 * cb + col); });
        }
#pragma unroll
        for (int i = 0; i < C::RBK; ++i) {
          const int rb = C::RBK * blk + i;
          if (rb < C::RB) {
            // phi(K)^T rows 16 rb .. 16 rb + 15 (k-order features), eight key tokens per lane
            const int kap = rb / 2, half = rb % 2;
            const int t0 = 32 * ks2 + 8 * g;
            auto pk_at = [&](int t, int col) -> const T* {
              const int f = 16 * half + col;  // feature offset within fragment kap
              return &sm.pk[par][t / 16][kap][16 * (f / 8) + t % 16][f % 8];
            };
            Frag<T> ka;
            load_tr4_at(ka, 0, lane, [&](int kk, int col) { return pk_at(t0 + kk, col); });
            load_tr4_at(ka, 4, lane, [&](int kk, int col) { return pk_at(t0 + 4 + kk, col); });
#pragma unroll
            for (int cb = 0; cb < C::CBT; ++cb) mma(sacc[i][cb], ka, bv[cb]);
            mma(zacc[i], ka, ones);
          }
        }
      }
      // phi(K) of the next chunk into the other buffer
      {
        Frag<T> ph[C::NF];
        feature_map(xa, c + 1, ph);
#pragma unroll
        for (int k = 0; k < C::NF; ++k) store8(&sm.pk[par ^ 1][blk][k][lane][0], ph[k]);
      }
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) xa[ks] = xb[ks];
      load_x(xb, c + 3);
    }
  }
}

template <typename T, int DH, int L, int MB, int DVT>
static hipError_t cs_run(const CausalArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((causal_kernel<T, DH, L, MB, DVT>), dim3(a.heads * a.dv_tiles), dim3(512), 0, s, a);
  return hipGetLastError();
}

// (dtype, d, L, projection blocks, value-column tile) combinations that are built.
#define LUNA_CS_CASES(X)      \
  X(float, 32, 8, 1, 32)      \
  X(float, 32, 2, 1, 32)      \
  X(float, 64, 8, 1, 32)      \
  X(__bf16, 32, 8, 1, 32)     \
  X(__bf16, 64, 8, 1, 64)     \
  X(__bf16, 64, 8, 2, 64)     \
  X(__bf16, 128, 8, 1, 64)    \
  X(__bf16, 128, 8, 2, 64)

template <typename T>
static constexpr Dt cs_dt_of() { return sizeof(T) == 2 ? Dt::BF16 : Dt::F32; }

bool causal_supported(Dt dt, int d, int L, int M, int* dv_tiles) {
  const int MB = (M + 15) / 16;
#define X(T_, D_, L_, MB_, DVT_)                                          \
  if (dt == cs_dt_of<T_>() && d == D_ && L == L_ && MB == MB_) {          \
    if (dv_tiles) *dv_tiles = D_ / DVT_;                                  \
    return true;                                                          \
  }
  LUNA_CS_CASES(X)
#undef X
  return false;
}

hipError_t launch_causal(Dt dt, int d, int L, int M, const CausalArgs& a, hipStream_t s) {
  const int MB = (M + 15) / 16;
#define X(T_, D_, L_, MB_, DVT_) \
  if (dt == cs_dt_of<T_>() && d == D_ && L == L_ && MB == MB_) return cs_run<T_, D_, L_, MB_, DVT_>(a, s);
  LUNA_CS_CASES(X)
#undef X
  return hipErrorInvalidValue;
}

}  // namespace luna
