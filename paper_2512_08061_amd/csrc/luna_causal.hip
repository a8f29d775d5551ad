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
// (head, tile of DVT value columns) and walks the chunks in order, keeping its
// slice of S in fp32 matrix-core accumulators; there is no cross-workgroup traffic.
//
// Per chunk:
//  A. waves 0-3 compute phi(Q) and waves 4-7 phi(K) of token block w % 4:
//     u^T = W X^T on the matrix cores (W fragments from LDS), one batched search of
//     the piecewise-linear table, L fused multiply-adds per projection.  The result
//     is k-order fragments (lane = token, 8 features) written to LDS.  Padded
//     projections and key tokens past n select the table's all-zero segment.
//  B. wave w answers query block i = (w < 4 ? w : 7 - w) (blocks i and 3 - i share a
//     SIMD, balancing the triangle) for value-column half w / 4:
//       P^T blocks j <= i = phi(K_j) phi(Q_i)^T, diagonal block masked; the
//       accumulators are directly the B operands of num^T += V^T P^T and of
//       den += 1^T P^T;  num^T += S^T phi(Q_i)^T, den += z^T phi(Q_i)^T from the
//       staged state;  out = num * (1 / (den + eps)).
//     Then S += phi(K_c)^T V_c for row blocks w, w + 8 of S (and z alongside).
//     V^T and phi(K)^T operands come from row-major LDS tiles through the gfx950
//     transpose read, so no data is stored transposed.
//  C. S and z are staged to LDS as A fragments for the next chunk.
// Two workgroup barriers per chunk; each wave's Q/K rows and the V tile are
// fetched into registers one chunk ahead.
#include "luna_device.hpp"
#include "luna_kernels.hpp"

namespace luna {

template <typename T, int DH, int L, int MB, int DVT>
struct CsCfg {
  static constexpr int KS = DH / 32;
  static constexpr int NF = (4 * MB * L + 7) / 8;   // k-order fragments over features
  static constexpr int FR = NF * 32;                // padded feature rows of S
  static constexpr int RB = FR / 16;                // row blocks of S
  static constexpr int RBW = (RB + 7) / 8;          // row blocks per wave
  static constexpr int CBT = DVT / 16;              // column blocks of the tile
  static constexpr int CBH = CBT / 2;               // column blocks per half
  static constexpr int SEGCAP = attn_seg_cap(L);
  static constexpr int VE = 16 / (int)sizeof(T);    // elements per 16-byte chunk
  static constexpr int VROW = DVT + VE;             // padded V-tile row (elements)
  static constexpr int VCH = 64 * DVT / VE;         // 16-byte chunks in a V tile
  static constexpr int NVC = (VCH + 511) / 512;     // per thread
  static_assert(CBT >= 2 && CBT % 2 == 0, "value tile must hold an even number of 16-column blocks");
};

template <typename T, int DH, int L, int MB, int DVT>
struct CsLds {
  using C = CsCfg<T, DH, L, MB, DVT>;
  PwlLds<C::SEGCAP> tab;
  alignas(16) T wfr[MB][C::KS][kWave][8];      // W as A fragments of u^T = W X^T
  alignas(16) T pq_tok[4][C::NF][kWave][8];    // phi(Q) fragments per token block
  alignas(16) T pk_tok[4][C::NF][kWave][8];    // phi(K) fragments per token block
  alignas(16) T vtile[64][C::VROW];            // V tile, row-major (token x column)
  alignas(16) T sst[C::CBT][C::NF][kWave][8];  // S_{c-1} as A fragments
  alignas(16) T zst[C::NF][4][8];              // z_{c-1} as A fragment slots per lane group
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

  // phase A role: side (0 = queries, 1 = keys) and token block
  const int side = wave / 4, tba = wave % 4;
  // phase B role: query block and value-column half
  const int qi = wave < 4 ? wave : 7 - wave, hh = wave / 4;
  const T* X = side ? K : Q;

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

  f32x4 sacc[C::RBW][C::CBT];
  f32x4 zacc[C::RBW];
#pragma unroll
  for (int i = 0; i < C::RBW; ++i) {
    zacc[i] = zero4();
#pragma unroll
    for (int cb = 0; cb < C::CBT; ++cb) sacc[i][cb] = zero4();
  }

  // one-chunk-ahead register fetch: this wave's X rows and its share of the V tile
  Frag<T> xn[C::KS];
  i32x4 vn[C::NVC];
  auto fetch = [&](int tc) {
    const int t = tc + 16 * tba + r;
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      if (t < n) load8(xn[ks], X + (size_t)t * DH + 32 * ks + 8 * g);
      else xn[ks].zero();
    }
#pragma unroll
    for (int q = 0; q < C::NVC; ++q) {
      const int cidx = tid + 512 * q;
      const int tt = cidx / (DVT / C::VE), cg = cidx % (DVT / C::VE);
      const int tv = tc + tt;
      if (cidx < C::VCH && tv < n) vn[q] = *reinterpret_cast<const i32x4*>(V + (size_t)tv * DH + c0 + cg * C::VE);
      else vn[q] = i32x4{0, 0, 0, 0};
    }
  };

  __syncthreads();
  const int tdepth = sm.tab.depth;
  const int zseg = sm.tab.zero_seg;
  const float tfloor = sm.tab.floor;
  const int nchunks = (n + 63) / 64;
  fetch(0);

  for (int c = 0; c < nchunks; ++c) {
    const int tc = 64 * c;
    // V tile of this chunk, row-major
#pragma unroll
    for (int q = 0; q < C::NVC; ++q) {
      const int cidx = tid + 512 * q;
      if (cidx < C::VCH) {
        const int tt = cidx / (DVT / C::VE), cg = cidx % (DVT / C::VE);
        *reinterpret_cast<i32x4*>(&sm.vtile[tt][cg * C::VE]) = vn[q];
      }
    }
    Frag<T> xc[C::KS];
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) xc[ks] = xn[ks];
    if (c + 1 < nchunks) fetch(tc + 64);

    // ---- A. feature map of this wave's (side, token block) ----
    {
      const bool tok_ok = tc + 16 * tba + r < n;
      float uu[4 * MB];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        f32x4 acc = zero4();
#pragma unroll
        for (int ks = 0; ks < C::KS; ++ks) {
          Frag<T> wa;
          load8(wa, &sm.wfr[mb][ks][lane][0]);
          mma(acc, wa, xc[ks]);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) uu[4 * mb + j] = acc[j] + brow[mb][j];
      }
      int sg[4 * MB];
      pwl_search(sm.tab, tdepth, uu, sg);
      const bool kill_tok = side && !tok_ok;  // key rows past n contribute nothing
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (!pok[mb][j] || kill_tok) sg[4 * mb + j] = zseg;
      Frag<T> ph[C::NF];
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
      T* dst = side ? &sm.pk_tok[tba][0][lane][0] : &sm.pq_tok[tba][0][lane][0];
#pragma unroll
      for (int k = 0; k < C::NF; ++k) store8(dst + (size_t)k * kWave * 8, ph[k]);
    }
    __syncthreads();

    // ---- B. query block qi, value columns of half hh ----
    {
      Frag<T> pq[C::NF];
#pragma unroll
      for (int k = 0; k < C::NF; ++k) load8(pq[k], &sm.pq_tok[qi][k][lane][0]);
      f32x4 pacc[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        pacc[j] = zero4();
        if (j <= qi) {
#pragma unroll
          for (int k = 0; k < C::NF; ++k) {
            Frag<T> ka;
            load8(ka, &sm.pk_tok[j][k][lane][0]);
            mma(pacc[j], ka, pq[k]);
          }
        }
      }
      // diagonal block: key token 16qi + 4g + jj after query token 16qi + r
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        if (4 * g + jj > r) {
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (j == qi) pacc[j][jj] = 0.0f;
        }

      f32x4 num[C::CBH], den = zero4();
#pragma unroll
      for (int cl = 0; cl < C::CBH; ++cl) num[cl] = zero4();
#pragma unroll
      for (int pr = 0; pr < 2; ++pr) {
        const int j0 = 2 * pr, j1 = 2 * pr + 1;
        if (j0 <= qi) {
          Frag<T> bp;
          const bool hi = j1 <= qi;
          bp.set2(0, pacc[j0][0], pacc[j0][1]);
          bp.set2(2, pacc[j0][2], pacc[j0][3]);
          bp.set2(4, hi ? pacc[j1][0] : 0.0f, hi ? pacc[j1][1] : 0.0f);
          bp.set2(6, hi ? pacc[j1][2] : 0.0f, hi ? pacc[j1][3] : 0.0f);
          mma(den, ones, bp);
#pragma unroll
          for (int cl = 0; cl < C::CBH; ++cl) {
            const int cb = hh * C::CBH + cl;
            Frag<T> va;
            load_tr4(va, 0, &sm.vtile[0][0], C::VROW, 16 * j0 + 4 * g, 16 * cb, lane);
            load_tr4(va, 4, &sm.vtile[0][0], C::VROW, 16 * j1 + 4 * g, 16 * cb, lane);
            mma(num[cl], va, bp);
          }
        }
      }
#pragma unroll
      for (int k = 0; k < C::NF; ++k) {
#pragma unroll
        for (int cl = 0; cl < C::CBH; ++cl) {
          Frag<T> sa;
          load8(sa, &sm.sst[hh * C::CBH + cl][k][lane][0]);
          mma(num[cl], sa, pq[k]);
        }
        Frag<T> za;
        load8(za, &sm.zst[k][g][0]);
        mma(den, za, pq[k]);
      }
      const int t = tc + 16 * qi + r;
      if (t < n) {
        const float rinv = 1.0f / (den[0] + a.eps);
        T* o = out + (size_t)t * DH + c0 + 4 * g;
#pragma unroll
        for (int cl = 0; cl < C::CBH; ++cl) {
          const int cb = hh * C::CBH + cl;
          store4(o + 16 * cb, num[cl][0] * rinv, num[cl][1] * rinv, num[cl][2] * rinv, num[cl][3] * rinv);
        }
      }
    }

    // ---- state update over the chunk's 64 key tokens ----
#pragma unroll
    for (int ks2 = 0; ks2 < 2; ++ks2) {
      Frag<T> bv[C::CBT];
#pragma unroll
      for (int cb = 0; cb < C::CBT; ++cb) {
        load_tr4(bv[cb], 0, &sm.vtile[0][0], C::VROW, 32 * ks2 + 8 * g, 16 * cb, lane);
        load_tr4(bv[cb], 4, &sm.vtile[0][0], C::VROW, 32 * ks2 + 8 * g + 4, 16 * cb, lane);
      }
#pragma unroll
      for (int i = 0; i < C::RBW; ++i) {
        const int rb = wave + 8 * i;
        if (rb < C::RB) {
          // phi(K)^T rows 16 rb .. 16 rb + 15 (k-order features), eight key tokens per lane
          const int kap = rb / 2, half = rb % 2;
          const int t0 = 32 * ks2 + 8 * g;
          auto pk_at = [&](int t, int col) -> const T* {
            const int f = 16 * half + col;  // feature offset within fragment kap
            return &sm.pk_tok[t / 16][kap][16 * (f / 8) + t % 16][f % 8];
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
    __syncthreads();
    // ---- C. stage S_c and z_c for the next chunk ----
#pragma unroll
    for (int i = 0; i < C::RBW; ++i) {
      const int rb = wave + 8 * i;
      if (rb < C::RB) {
        const int k = rb / 2, gp = 2 * (rb % 2) + g / 2, e0 = 4 * (g % 2);
#pragma unroll
        for (int cb = 0; cb < C::CBT; ++cb)
          store4(&sm.sst[cb][k][16 * gp + r][e0], sacc[i][cb][0], sacc[i][cb][1], sacc[i][cb][2], sacc[i][cb][3]);
        if (r == 0) store4(&sm.zst[k][gp][e0], zacc[i][0], zacc[i][1], zacc[i][2], zacc[i][3]);
      }
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
