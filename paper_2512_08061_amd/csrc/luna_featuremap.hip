// luna_featuremap.hip -- phi(x) of eq. (11) of Section 3.2 for every row of X.
//
// One wave handles 16 rows of one head.  The projections are computed transposed,
// u^T = W X^T, on the matrix cores: A = W (row = projection, k = d), B = X^T
// (column = row of X, k = d), so each lane ends up holding four projections
// 16mb + 4g + j (j = 0..3) of the row r = lane % 16.  The channel functions are
// evaluated in registers from the piecewise-linear table and the L outputs of each
// (row, projection) are stored contiguously at feature i*L + l.
#include "luna_device.hpp"
#include "luna_kernels.hpp"

namespace luna {

constexpr int kFmCopyPerBlock = 1024;  // floats per copying workgroup (four per thread)

// HOLD: at most four 16-projection blocks, whose W fragments and biases stay in
// registers for every item of the parameter set; maps with more blocks reload them
// per group (held across items they would cost the registers that keep those maps'
// occupancy).
template <typename Tin, typename Tout, int DH, int L, bool HOLD>
__global__ __launch_bounds__(256) void featuremap_kernel(FeatureMapArgs a) {
  constexpr int KS = DH / 32;
  __shared__ PwlLds<L, nseg_cap(L, kFmSegBytes)> tab;

  if ((int)blockIdx.x >= a.map_grid) {  // (uniform) a copying workgroup: kFmCopyPerBlock floats
    const int64_t base = (int64_t)(blockIdx.x - a.map_grid) * kFmCopyPerBlock + threadIdx.x;
    float v[kFmCopyPerBlock / 256];
#pragma unroll
    for (int j = 0; j < kFmCopyPerBlock / 256; ++j) {
      const int64_t i = base + 256 * j;
      v[j] = i < a.copy_n ? a.copy_src[i] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < kFmCopyPerBlock / 256; ++j) {
      const int64_t i = base + 256 * j;
      if (i < a.copy_n) a.copy_dst[i] = v[j];
    }
    return;
  }
  const int tiles_per_head = (int)((a.rows_per_head + 63) / 64);
  // work items: 64-row tiles of every head; with a second input the items double and
  // the second half maps X2 into out2.  A workgroup takes items blockIdx.x,
  // blockIdx.x + map_grid, ..., so that its table copy serves many tiles.
  const int64_t per_input = a.heads * tiles_per_head;
  const int64_t items = per_input * (a.X2 != nullptr ? 2 : 1);
  const int wave = wave_id(), lane = threadIdx.x % kWave;
  const int g = lane / 16, r = lane % 16;
  const int64_t n = a.rows_per_head;
  const int M = a.phi.M;
  const int D = M * L;
  // projections go in groups of four 16-projection blocks (W fragments of one group
  // in registers; with at most four blocks they stay there for every item of the
  // parameter set)
  constexpr int kMaxMB = 4;
  const int MB = (M + 15) / 16;
  // item -> its input, output, parameter set and this lane's row (B column)
  struct Item {
    const Tin* X;
    Tout* out;
    int hset;
    bool row_ok;
  };
  auto locate = [&](int64_t item) {
    int64_t bid = item;
    const void* Xsrc = a.X;
    void* Odst = a.out;
    if (bid >= per_input) {
      bid -= per_input;
      Xsrc = a.X2;
      Odst = a.out2;
    }
    const int64_t head = bid / tiles_per_head;
    const int tile = (int)(bid - head * tiles_per_head);
    const int64_t t = (int64_t)tile * 64 + wave * 16 + r;
    Item it;
    it.row_ok = t < n;
    it.hset = a.phi.per_head ? (int)(head % a.H) : 0;
    it.X = reinterpret_cast<const Tin*>(Xsrc) + (head * n + (it.row_ok ? t : 0)) * DH;
    it.out = reinterpret_cast<Tout*>(Odst) + (head * n + (it.row_ok ? t : 0)) * (int64_t)D;
    return it;
  };
  auto load_row = [&](Frag<Tin> (&xf)[KS], const Item& it) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (it.row_ok) load8(xf[ks], it.X + 32 * ks + 8 * g);
      else xf[ks].zero();
    }
  };
  int loaded = -1;
  {
    int wset = -1;
    Frag<Tin> wfr[kMaxMB][KS];
    float bz[kMaxMB][4];
    for (int64_t item = blockIdx.x; item < items; item += a.map_grid) {
      const Item cur = locate(item);
      const int hset = cur.hset;
      const bool row_ok = cur.row_ok;
      Tout* out = cur.out;
      const Tin* W = reinterpret_cast<const Tin*>(a.phi.W) + (size_t)hset * M * DH;
      const float* bias = a.phi.b + (size_t)hset * M;
      // the row, W fragments and biases are fetched before the table, so that their
      // loads overlap its copy
      Frag<Tin> xf[KS];
      load_row(xf, cur);
      for (int mg = 0; mg < MB; mg += kMaxMB) {
        if (!HOLD || hset != wset) {  // (uniform)
#pragma unroll
          for (int mbl = 0; mbl < kMaxMB; ++mbl) {
            const int mb = mg + mbl;
            const int prow = 16 * mb + r;  // W row this lane feeds to the A operand
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
              if (mb < MB && prow < M) load8(wfr[mbl][ks], W + (size_t)prow * DH + 32 * ks + 8 * g);
              else wfr[mbl][ks].zero();
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const int i = 16 * mb + 4 * g + j;  // projection held in acc[j]
              bz[mbl][j] = (mb < MB && i < M) ? bias[i] : 0.0f;
            }
          }
          wset = hset;
        }
        if (mg == 0 && hset != loaded) {  // (uniform) a workgroup loads a table once per parameter set it meets
          __syncthreads();                // every wave is done with the previous table
          pwl_load(tab, a.phi.tables + (size_t)hset * kTableBytes);
          __syncthreads();
          loaded = hset;
        }
        const int steps = __builtin_amdgcn_readfirstlane(tab.steps);
        const float floor = tab.floor;

        // the group's projections, then one search over all of them, so that the
        // searches' dependent LDS reads overlap
        float uu[4 * kMaxMB];
#pragma unroll
        for (int mbl = 0; mbl < kMaxMB; ++mbl) {
          f32x4 acc = zero4();
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) mma(acc, wfr[mbl][ks], xf[ks]);
#pragma unroll
          for (int j = 0; j < 4; ++j) uu[4 * mbl + j] = acc[j] + bz[mbl][j];
        }
        int sg[4 * kMaxMB];
        pwl_search(tab, steps, uu, sg);
#pragma unroll
        for (int mbl = 0; mbl < kMaxMB; ++mbl) {
          const int mb = mg + mbl;
          if (mb >= MB || !row_ok) break;
          const int i0 = 16 * mb + 4 * g;  // projections i0 .. i0 + 3 of this lane
          float y[4][L];
#pragma unroll
          for (int j = 0; j < 4; ++j) pwl_channels<L>(tab, sg[4 * mbl + j], floor, uu[4 * mbl + j], y[j]);
          Tout* o = out + i0 * L;
          if (i0 + 3 < M) {  // the four projections' 4 L features are contiguous
#pragma unroll
            for (int q = 0; q < L; ++q) {
              const float* f = &y[0][0] + 4 * q;  // features 4 q .. 4 q + 3 of the four
              store4(o + 4 * q, f[0], f[1], f[2], f[3]);
            }
          } else {
#pragma unroll
            for (int j = 0; j < 4; ++j)
              if (i0 + j < M)
#pragma unroll
                for (int l = 0; l < L; ++l) o[j * L + l] = (Tout)y[j][l];
          }
        }
      }
    }
  }
}

// As many mapping workgroups as the device holds at once (registers and LDS table
// permitting), queried once per kernel (the kernel is a template argument, so that
// every kernel has its own cached count); more items loop, so that no second round of
// workgroups starts late.  The copying workgroups, if any, follow them in the grid.
template <auto Kernel>
static void fm_launch(int64_t items, const FeatureMapArgs& args, hipStream_t s) {
  static const int resident = []() {
    int per_cu = 0, dev = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, Kernel, 256, 0) != hipSuccess || per_cu < 1) per_cu = 1;
    if (hipGetDevice(&dev) != hipSuccess) dev = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) cus = 256;
    return per_cu * cus;
  }();
  FeatureMapArgs a = args;
  a.map_grid = (int)(items < resident ? items : resident);
  const int64_t copy_blocks = a.copy_n > 0 ? (a.copy_n + kFmCopyPerBlock - 1) / kFmCopyPerBlock : 0;
  hipLaunchKernelGGL(Kernel, dim3((unsigned)(a.map_grid + copy_blocks)), dim3(256), 0, s, a);
}

template <typename Tin, typename Tout, int DH>
static hipError_t fm_dispatch_L(int L, const FeatureMapArgs& a, hipStream_t s) {
  const int64_t tiles = (a.rows_per_head + 63) / 64;
  const int64_t items = a.heads * tiles * (a.X2 != nullptr ? 2 : 1);
  const bool hold = a.phi.M <= 64;  // at most four 16-projection blocks
#define LUNA_FM_LAUNCH(L_)                                                                  \
  if (hold) fm_launch<featuremap_kernel<Tin, Tout, DH, L_, true>>(items, a, s);             \
  else fm_launch<featuremap_kernel<Tin, Tout, DH, L_, false>>(items, a, s);
  switch (L) {
    case 1: LUNA_FM_LAUNCH(1) break;
    case 2: LUNA_FM_LAUNCH(2) break;
    case 4: LUNA_FM_LAUNCH(4) break;
    case 8: LUNA_FM_LAUNCH(8) break;
    case 16: LUNA_FM_LAUNCH(16) break;
    default: return hipErrorInvalidValue;
  }
#undef LUNA_FM_LAUNCH
  return hipGetLastError();
}

template <typename Tin, typename Tout>
static hipError_t fm_dispatch_d(int d, int L, const FeatureMapArgs& a, hipStream_t s) {
  switch (d) {
    case 32: return fm_dispatch_L<Tin, Tout, 32>(L, a, s);
    case 64: return fm_dispatch_L<Tin, Tout, 64>(L, a, s);
    case 128: return fm_dispatch_L<Tin, Tout, 128>(L, a, s);
    default: return hipErrorInvalidValue;
  }
}

bool featuremap_supported(Dt, int d, int L, int M) {
  const bool dok = d == 32 || d == 64 || d == 128;
  const bool lok = L == 1 || L == 2 || L == 4 || L == 8 || L == 16;
  return dok && lok && M >= 1 && M <= 256 && M * L <= 256;
}

hipError_t launch_featuremap(Dt in_dt, Dt out_dt, int d, int L, const FeatureMapArgs& a, hipStream_t s) {
  if (in_dt == Dt::BF16)
    return out_dt == Dt::BF16 ? fm_dispatch_d<__bf16, __bf16>(d, L, a, s) : fm_dispatch_d<__bf16, float>(d, L, a, s);
  return out_dt == Dt::BF16 ? fm_dispatch_d<float, __bf16>(d, L, a, s) : fm_dispatch_d<float, float>(d, L, a, s);
}

}  // namespace luna
