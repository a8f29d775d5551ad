// luna_causal.hip -- causal (streaming) LUNA attention as a chunked prefix scan.
//
// out_t = phi(q_t)^T S_t / (phi(q_t)^T z_t + eps) with S_t, z_t summed over s <= t.
// Tokens are processed in chunks of 64; within chunk c (rows of the chunk t, columns s):
//
//   P      = tril(phi(Q_c) phi(K_c)^T)              (diagonal included)
//   num    = P V_c + phi(Q_c) S_{c-1},   den = P 1 + phi(Q_c) z_{c-1}
//   S_c    = S_{c-1} + phi(K_c)^T V_c,   z_c = z_{c-1} + phi(K_c)^T 1
//
// which regroups the prefix sums exactly.  One workgroup owns one (head, tile of
// DVT value columns) and walks the chunks in order, keeping its slice of S in fp32
// matrix-core accumulators and z alongside; there is no cross-workgroup traffic.
//
// Within a chunk wave w owns query/key token block w (16 tokens):
//  1. u^T = W Q^T and u^T = W K^T (A = W fragments from LDS), psi -> phi(Q_w), phi(K_w)
//     as k-order fragments (lane = token, 8 features), see luna_noncausal.hip.
//  2. phi(K_w) goes to LDS twice: as fragments (for other waves' P blocks) and
//     transposed, feature x token (for the state update).
//  3. P^T blocks (j <= w) = phi(K_j) phi(Q_w)^T; the diagonal block is masked.  The
//     accumulators are already B fragments of num^T += V^T P^T (k = key token);
//     den += 1^T P^T with an all-ones A operand.
//  4. num^T += S^T phi(Q_w)^T and den += z^T phi(Q_w)^T, S and z read from LDS as
//     A fragments (staged at the end of the previous chunk, bf16 for bf16 calls).
//  5. out = num * (1 / (den + eps)).
//  6. S += phi(K_c)^T V_c over the chunk (wave w updates row blocks w, w+4, ...),
//     then S and z are staged to LDS for the next chunk.
// Two workgroup barriers per chunk; V and the next chunk's Q/K rows are fetched into
// registers one chunk ahead.
#include "luna_device.hpp"
#include "luna_kernels.hpp"

namespace luna {

template <typename T, int DH, int L, int MB, int DVT>
struct CsCfg {
  static constexpr int KS = DH / 32;
  static constexpr int NF = (4 * MB * L + 7) / 8;   // k-order fragments over features
  static constexpr int FR = NF * 32;                // padded feature rows of S
  static constexpr int RB = FR / 16;                // row blocks of S
  static constexpr int RBW = (RB + 3) / 4;          // row blocks per wave
  static constexpr int CBT = DVT / 16;              // column blocks of the tile
  static constexpr int SEGCAP = attn_seg_cap(L);
  static constexpr int VE = 16 / (int)sizeof(T);
  static constexpr int TROW = 64 + VE;              // token-row length in LDS (padded)
  static constexpr int NVC = 64 * (DVT / VE) / 256; // V 16-byte chunks per thread per chunk
  static_assert(NVC >= 1, "value tile too narrow");
};

template <typename T, int DH, int L, int MB, int DVT>
struct CsLds {
  using C = CsCfg<T, DH, L, MB, DVT>;
  PwlLds<C::SEGCAP> tab;
  alignas(16) T wfr[MB][C::KS][kWave][8];   // W as A fragments of u^T = W X^T
  alignas(16) T pk_tok[4][C::NF][kWave][8]; // phi(K) fragments per token block
  alignas(16) T pk_t[C::FR][C::TROW];       // phi(K)^T: k-order feature x token
  alignas(16) T vt[DVT][C::TROW];           // V^T tile: value column x token
  alignas(16) T sst[C::CBT][C::NF][kWave][8];  // S_{c-1} as A fragments
  alignas(16) T zst[C::NF][4][8];              // z_{c-1} as A fragment slots per lane group
};

template <typename T, int DH, int L, int MB, int DVT>
__global__ __launch_bounds__(256, 1) void causal_kernel(CausalArgs a) {
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

  // W fragments into LDS; S and z start at zero
  for (int i = tid; i < MB * C::KS * kWave; i += 256) {
    const int l = i % kWave, ks = (i / kWave) % C::KS, mb = i / (kWave * C::KS);
    const int p = 16 * mb + l % 16;
    Frag<T> f;
    if (p < M) load8(f, W + (size_t)p * DH + 32 * ks + 8 * (l / 16));
    else f.zero();
    store8(&sm.wfr[mb][ks][l][0], f);
  }
  for (int i = tid; i < C::CBT * C::NF * kWave; i += 256) {
    Frag<T> f;
    f.zero();
    store8(&sm.sst[0][0][0][0] + (size_t)i * 8, f);
  }
  for (int i = tid; i < C::NF * 4; i += 256) {
    Frag<T> f;
    f.zero();
    store8(&sm.zst[0][0][0] + (size_t)i * 8, f);
  }
  float brow[MB][4];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = 16 * mb + 4 * g + j;
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

  // one-chunk-ahead register fetch
  Frag<T> qn[C::KS], kn[C::KS];
  i32x4 vn[C::NVC];
  auto fetch = [&](int tc) {
    const int t = tc + 16 * wave + r;
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      if (t < n) {
        load8(qn[ks], Q + (size_t)t * DH + 32 * ks + 8 * g);
        load8(kn[ks], K + (size_t)t * DH + 32 * ks + 8 * g);
      } else {
        qn[ks].zero();
        kn[ks].zero();
      }
    }
#pragma unroll
    for (int q = 0; q < C::NVC; ++q) {
      const int cidx = tid + 256 * q;
      const int tt = cidx / (DVT / C::VE), cg = cidx % (DVT / C::VE);
      const int tv = tc + tt;
      if (tv < n) vn[q] = *reinterpret_cast<const i32x4*>(V + (size_t)tv * DH + c0 + cg * C::VE);
      else vn[q] = i32x4{0, 0, 0, 0};
    }
  };

  __syncthreads();
  const int tdepth = sm.tab.depth;
  const float tfloor = sm.tab.floor;
  const int nchunks = (n + 63) / 64;
  fetch(0);

  for (int c = 0; c < nchunks; ++c) {
    const int tc = 64 * c;
    // V^T tile of this chunk
#pragma unroll
    for (int q = 0; q < C::NVC; ++q) {
      const int cidx = tid + 256 * q;
      const int tt = cidx / (DVT / C::VE), cg = cidx % (DVT / C::VE);
      const T* e = reinterpret_cast<const T*>(&vn[q]);
#pragma unroll
      for (int x = 0; x < C::VE; ++x) sm.vt[cg * C::VE + x][tt] = e[x];
    }
    Frag<T> qc[C::KS], kc[C::KS];
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      qc[ks] = qn[ks];
      kc[ks] = kn[ks];
    }
    if (c + 1 < nchunks) fetch(tc + 64);

    // 1. projections and channel functions of this wave's 16 tokens
    const bool k_ok = tc + 16 * wave + r < n;
    Frag<T> pq[C::NF], pk[C::NF];
#pragma unroll
    for (int k = 0; k < C::NF; ++k) {
      pq[k].zero();
      pk[k].zero();
    }
    float uu[8 * MB];  // q projections at [4mb + j], k projections at [4MB + 4mb + j]
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      f32x4 aq = zero4(), ak = zero4();
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) {
        Frag<T> wa;
        load8(wa, &sm.wfr[mb][ks][lane][0]);
        mma(aq, wa, qc[ks]);
        mma(ak, wa, kc[ks]);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        uu[4 * mb + j] = aq[j] + brow[mb][j];
        uu[4 * MB + 4 * mb + j] = ak[j] + brow[mb][j];
      }
    }
    int sg[8 * MB];
    pwl_search(sm.tab, tdepth, uu, sg);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bool pok = 16 * mb + 4 * g + j < M;
        float yq[L], yk[L];
        pwl_channels<L>(sm.tab, sg[4 * mb + j], tfloor, uu[4 * mb + j], yq);
        pwl_channels<L>(sm.tab, sg[4 * MB + 4 * mb + j], tfloor, uu[4 * MB + 4 * mb + j], yk);
#pragma unroll
        for (int l = 0; l < L; ++l) {
          const int p = (mb * 4 + j) * L + l;
          pq[p / 8].set(p % 8, pok ? yq[l] : 0.0f);
          pk[p / 8].set(p % 8, (pok && k_ok) ? yk[l] : 0.0f);
        }
      }
    }
    // 2. phi(K_w) to LDS
#pragma unroll
    for (int k = 0; k < C::NF; ++k) {
      store8(&sm.pk_tok[wave][k][lane][0], pk[k]);
#pragma unroll
      for (int e = 0; e < 8; ++e) sm.pk_t[32 * k + 8 * g + e][16 * wave + r] = pk[k].v[e];
    }
    __syncthreads();

    // 3. intra-chunk block
    f32x4 pacc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      pacc[j] = zero4();
      if (j <= wave) {
#pragma unroll
        for (int k = 0; k < C::NF; ++k) {
          if (j == wave) {
            mma(pacc[j], pk[k], pq[k]);
          } else {
            Frag<T> ka;
            load8(ka, &sm.pk_tok[j][k][lane][0]);
            mma(pacc[j], ka, pq[k]);
          }
        }
      }
    }
#pragma unroll
    for (int jj = 0; jj < 4; ++jj)
      if (4 * g + jj > r) {
        // diagonal block: key token 16w + 4g + jj after query token 16w + r
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (j == wave) pacc[j][jj] = 0.0f;
      }

    f32x4 num[C::CBT], den = zero4();
#pragma unroll
    for (int cb = 0; cb < C::CBT; ++cb) num[cb] = zero4();
#pragma unroll
    for (int pr = 0; pr < 2; ++pr) {
      const int j0 = 2 * pr, j1 = 2 * pr + 1;
      if (j0 <= wave) {
        Frag<T> bp;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          bp.set(e, pacc[j0][e]);
          bp.set(4 + e, j1 <= wave ? pacc[j1][e] : 0.0f);
        }
        mma(den, ones, bp);
#pragma unroll
        for (int cb = 0; cb < C::CBT; ++cb) {
          Frag<T> va;
          load4(va, 0, &sm.vt[16 * cb + r][16 * j0 + 4 * g]);
          load4(va, 4, &sm.vt[16 * cb + r][16 * j1 + 4 * g]);
          mma(num[cb], va, bp);
        }
      }
    }
    // 4. carried state
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
    // 5. output rows of this wave
    {
      const int t = tc + 16 * wave + r;
      if (t < n) {
        const float rinv = 1.0f / (den[0] + a.eps);
        T* o = out + (size_t)t * DH + c0 + 4 * g;
#pragma unroll
        for (int cb = 0; cb < C::CBT; ++cb)
          store4(o + 16 * cb, num[cb][0] * rinv, num[cb][1] * rinv, num[cb][2] * rinv, num[cb][3] * rinv);
      }
    }
    // 6. state update over the chunk's 64 key tokens
#pragma unroll
    for (int ks2 = 0; ks2 < 2; ++ks2) {
      Frag<T> bv[C::CBT];
#pragma unroll
      for (int cb = 0; cb < C::CBT; ++cb) load8(bv[cb], &sm.vt[16 * cb + r][32 * ks2 + 8 * g]);
#pragma unroll
      for (int i = 0; i < C::RBW; ++i) {
        const int rb = wave + 4 * i;
        if (rb < C::RB) {
          Frag<T> ka;
          load8(ka, &sm.pk_t[16 * rb + r][32 * ks2 + 8 * g]);
#pragma unroll
          for (int cb = 0; cb < C::CBT; ++cb) mma(sacc[i][cb], ka, bv[cb]);
          mma(zacc[i], ka, ones);
        }
      }
    }
    __syncthreads();
    // stage S_c and z_c for the next chunk
#pragma unroll
    for (int i = 0; i < C::RBW; ++i) {
      const int rb = wave + 4 * i;
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
  hipLaunchKernelGGL((causal_kernel<T, DH, L, MB, DVT>), dim3(a.heads * a.dv_tiles), dim3(256), 0, s, a);
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
