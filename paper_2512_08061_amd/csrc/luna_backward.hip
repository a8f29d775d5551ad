// luna_backward.hip -- gradients of LUNA attention (training the feature map end to
// end and fine-tuning converted models).
//
// For a loss L with upstream gradient dO = dL/dout, with num = phi(Q) S, den = phi(Q) z
// + eps and out = num / den per row (eq. (9) of Section 3.1; prefix states for the
// causal form), the chain rule gives, per row t and with G_t = [dnum_t | dden_t],
//   dnum_t = dO_t / den_t,  dden_t = -(dO_t . num_t) / den_t^2,
//   dphi(q_t) = G_t [S_t | z_t]^T,
//   [dS | dz] = phi(Q)^T G  (non-causal; causal: suffix sums over t >= s),
//   dphi(k_s) = [v_s | 1] [dS_s | dz_s]^T,  dv_s = dS_s^T phi(k_s),
// and through the feature map phi_{iL+l} = relu(y_l(u_i)) / sqrt(M), u = x W^T + b,
// y_l(u) = g_l + sum_k f_lk relu(a_lk u + c_lk) (ReLU'(0) = 0).
//
// The causal form is taken in chunks of C tokens: with the exclusive prefix state
// [S_c | z_c] before chunk c and P_c = tril(phi(Q_c) phi(K_c)^T),
//   [num | den - eps]_c = phi(Q_c) [S_c | z_c] + P_c [V_c | 1],
//   dphi(Q_c) = G_c [S_c | z_c]^T + R_c phi(K_c),   R_c = tril(G_c [V_c | 1]^T),
// and with the exclusive suffix state [dS_c | dz_c] after chunk c,
//   dphi(K_c) = [V_c | 1] [dS_c | dz_c]^T + R_c^T phi(Q_c),
//   dV_c = phi(K_c) dS_c + P_c^T dnum_c,
// an exact regrouping of the sums.  The non-causal form is the same with the total
// state in place of the prefix and suffix states and no intra-chunk terms (its
// chunks only split the sums over tokens among more workgroups).
//
// Kernels (all arithmetic in fp32):
//   bwd_pack_kernel     V -> [V | 1] in fp32;
//   bwd_gemm_kernel     batched C (+)= A B over (head, chunk) with strided operands, a
//                       lower-triangular output mask and ragged last chunks;
//   bwd_scan_kernel     exclusive prefix or suffix sums of the per-chunk states (or, for
//                       the non-causal form, split into chunks only for parallelism,
//                       their total);
//   bwd_g_kernel        [num | den - eps] -> G = [dnum | dden];
//   bwd_packw_kernel    [W | b] in fp32: u = [x | 1] [W | b]^T, dx = du [W | b] (first d
//                       columns), [dW | db] = du^T [x | 1] are GEMMs;
//   bwd_phi_kernel      dphi -> du, one thread per (row, projection): the slopes of the
//                       piecewise-linear channel functions, zero where the output ReLU
//                       is off, and per workgroup the (segment, channel) moments sum dy
//                       and sum dy u of the channel outputs' gradients;
//   bwd_dw_kernel       [dW | db] summed over the (batch, head) products;
//   bwd_reduce_kernel   the partials summed over workgroups (fp64);
//   bwd_prefix_kernel   exclusive prefix sums of the moments over segments, per channel;
//   bwd_mlp_kernel      the channel-MLP parameter gradients from the moments: unit k
//                       is on exactly on the segments above (a_k > 0) or below
//                       (a_k < 0) its breakpoint, where h_k = a_k u + c_k, so
//                       dfc2_lk = a_k sum_on dy_l u + c_k sum_on dy_l,
//                       dfc1_(l)k = f_lk sum_on dy_l u, dfc1_b likewise, dfc2_b_l = sum dy_l.
//
// The same pack, GEMM and scan kernels carry the forward pass of the shapes that have
// no fused kernel (any d, L and M the feature-map kernel takes: one channel per
// projection with M up to 256, fp32 at d = 128, ...), in fp32 throughout, with two more:
//   fwd_out_kernel      [num | den - eps] -> out = num / den in the call's dtype;
//   fwd_export_kernel   the total [S | z] of a head into (or added to) the caller's S, z.
#include <algorithm>

#include "luna_device.hpp"
#include "luna_kernels.hpp"

namespace luna {

namespace {

// ---------------------------------------------------------------------------
// [V | 1] in fp32
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void bwd_pack_kernel(const T* __restrict__ V, float* __restrict__ Vx, int64_t rows,
                                                       int d) {
  const int64_t total = rows * (d + 1);
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / (d + 1);
    const int c = (int)(i - r * (d + 1));
    Vx[i] = c < d ? (float)V[r * d + c] : 1.0f;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void bwd_convert_kernel(const float* __restrict__ src, T* __restrict__ dst,
                                                          int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = (T)src[i];
}

// ---------------------------------------------------------------------------
// batched strided GEMM on the fp32 matrix cores: 64 x 64 output tiles, four waves
// of 32 x 32 (2 x 2 blocks of 16 x 16), 32-deep k slices through LDS, the next slice
// read into registers during the current slice's products.  A tile is kept
// row-major (i, k) and B transposed (j, k), so that a lane's fragment -- row (or
// column) lane % 16, k = 8 (lane / 16) + e for e < 8 -- is two 16-byte reads.  Tile
// loads let consecutive threads walk the operand's unit-stride index.
// ---------------------------------------------------------------------------
constexpr int kGT = 64, kGK = 32, kGP = kGK + 4;  // tile, k slice, LDS row (floats)

__global__ __launch_bounds__(256) void bwd_gemm_kernel(BwdGemm g) {
  __shared__ __attribute__((aligned(16))) float As[kGT][kGP];
  __shared__ __attribute__((aligned(16))) float Bt[kGT][kGP];
  const int bz = blockIdx.z;
  const int h = bz / g.chunks, c = bz - h * g.chunks;
  const int rows_left = g.seq - c * g.chunk;  // tokens of this chunk (ragged last chunk)
  const int Mv = g.m_chunk ? min(g.M, rows_left) : g.M;
  const int Nv = g.n_chunk ? min(g.N, rows_left) : g.N;
  const int Kv = g.k_chunk ? min(g.K, rows_left) : g.K;
  const float* A = g.A + h * g.sAh + c * g.sAc;
  const float* B = g.B + h * g.sBh + c * g.sBc;
  float* C = g.C + h * g.sCh + c * g.sCc;
  const int i0 = blockIdx.y * kGT, j0 = blockIdx.x * kGT;
  if (i0 >= Mv || j0 >= Nv) return;  // (uniform) tile outside this chunk's rows
  const int tid = threadIdx.x, lane = tid % kWave, wave = wave_id();
  const int grp = lane / 16, r = lane % 16;
  const int wi = 32 * (wave / 2), wj = 32 * (wave % 2);  // this wave's 32 x 32 sub-tile
  const bool a_krow = g.sAk == 1, b_jrow = g.sBj == 1;   // unit stride along k (A) or j (B)
  f32x4 acc[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y) acc[x][y] = zero4();
  // The next k slice is read into registers while the matrix cores work on the current
  // one from LDS, so that global-load latency overlaps the products.
  constexpr int PER = (kGK * kGT) / 256;  // elements of each operand per thread and slice
  float ra[PER], rb[PER];
  auto load_slice = [&](int k0) {
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int idx = tid + 256 * e;
      int ii, kk;
      if (a_krow) { kk = idx % kGK; ii = idx / kGK; }
      else { ii = idx % kGT; kk = idx / kGT; }
      const int ia = i0 + ii, ka = k0 + kk;
      ra[e] = (ka < Kv && ia < Mv) ? A[ia * g.sAi + ka * g.sAk] : 0.0f;
      int jj, kb;
      if (b_jrow) { jj = idx % kGT; kb = idx / kGT; }
      else { kb = idx % kGK; jj = idx / kGK; }
      const int jb = j0 + jj, kbb = k0 + kb;
      rb[e] = (kbb < Kv && jb < Nv) ? B[kbb * g.sBk + jb * g.sBj] : 0.0f;
    }
  };
  auto store_slice = [&]() {
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int idx = tid + 256 * e;
      int ii, kk;
      if (a_krow) { kk = idx % kGK; ii = idx / kGK; }
      else { ii = idx % kGT; kk = idx / kGT; }
      As[ii][kk] = ra[e];
      int jj, kb;
      if (b_jrow) { jj = idx % kGT; kb = idx / kGT; }
      else { kb = idx % kGK; jj = idx / kGK; }
      Bt[jj][kb] = rb[e];
    }
  };
  load_slice(0);
  for (int k0 = 0; k0 < Kv; k0 += kGK) {
    store_slice();
    __syncthreads();
    if (k0 + kGK < Kv) load_slice(k0 + kGK);
    Frag<float> af[2], bf[2];
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      const float4* pa = reinterpret_cast<const float4*>(&As[wi + 16 * x + r][8 * grp]);
      const float4* pb = reinterpret_cast<const float4*>(&Bt[wj + 16 * x + r][8 * grp]);
      const float4 a0 = pa[0], a1 = pa[1], b0 = pb[0], b1 = pb[1];
      af[x].v[0] = a0.x; af[x].v[1] = a0.y; af[x].v[2] = a0.z; af[x].v[3] = a0.w;
      af[x].v[4] = a1.x; af[x].v[5] = a1.y; af[x].v[6] = a1.z; af[x].v[7] = a1.w;
      bf[x].v[0] = b0.x; bf[x].v[1] = b0.y; bf[x].v[2] = b0.z; bf[x].v[3] = b0.w;
      bf[x].v[4] = b1.x; bf[x].v[5] = b1.y; bf[x].v[6] = b1.z; bf[x].v[7] = b1.w;
    }
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int y = 0; y < 2; ++y) mma(acc[x][y], af[x], bf[y]);
    __syncthreads();
  }
  // acc[x][y] holds rows 4 grp + q (q < 4), column r of block (x, y)
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int i = i0 + wi + 16 * x + 4 * grp + q, j = j0 + wj + 16 * y + r;
        if (i >= Mv || j >= Nv) continue;
        float v = (g.lower && j > i) ? 0.0f : acc[x][y][q];
        float* pc = C + i * g.sCi + j * g.sCj;
        if (g.accumulate) v += *pc;
        *pc = v;
      }
}

// ---------------------------------------------------------------------------
// exclusive prefix (forward) or suffix (backward) sums over chunks, in place
// ---------------------------------------------------------------------------
// mode 0: exclusive prefix, 1: exclusive suffix, 2: the total in every chunk
__global__ __launch_bounds__(256) void bwd_scan_kernel(float* X, int heads, int chunks, int64_t elems, int mode) {
  const int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int h = blockIdx.y;
  if (e >= elems || h >= heads) return;
  float* base = X + (int64_t)h * chunks * elems + e;
  float run = 0.0f;
  for (int i = 0; i < chunks; ++i) {
    const int c = mode == 1 ? chunks - 1 - i : i;
    const float v = base[(int64_t)c * elems];
    if (mode != 2) base[(int64_t)c * elems] = run;
    run += v;
  }
  if (mode == 2)
    for (int c = 0; c < chunks; ++c) base[(int64_t)c * elems] = run;
}

// ---------------------------------------------------------------------------
// [num | den - eps] -> [dnum | dden], one wave per row
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void bwd_g_kernel(float* __restrict__ Y, const T* __restrict__ dO, int64_t rows,
                                                    int d, float eps) {
  const int lane = threadIdx.x % kWave;
  const int64_t r = blockIdx.x * (int64_t)(blockDim.x / kWave) + threadIdx.x / kWave;
  if (r >= rows) return;
  float* y = Y + r * (d + 1);
  const T* go = dO + r * d;
  const float den = y[d] + eps;
  float dot = 0.0f;
  for (int c = lane; c < d; c += kWave) dot = fmaf((float)go[c], y[c], dot);
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) dot += __shfl_xor(dot, o, kWave);
  const float inv = 1.0f / den;
  for (int c = lane; c < d; c += kWave) y[c] = (float)go[c] * inv;
  if (lane == 0) y[d] = -dot * inv * inv;
}

// ---------------------------------------------------------------------------
// forward readout of the generic path: out = num / (den - eps + eps), one wave per row
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void fwd_out_kernel(const float* __restrict__ Y, T* __restrict__ out, int64_t rows,
                                                      int d, float eps) {
  const int lane = threadIdx.x % kWave;
  const int64_t r = blockIdx.x * (int64_t)(blockDim.x / kWave) + threadIdx.x / kWave;
  if (r >= rows) return;
  const float* y = Y + r * (d + 1);
  const float inv = 1.0f / (y[d] + eps);
  for (int c = lane; c < d; c += kWave) out[r * d + c] = (T)(y[c] * inv);
}

// [S | z] of each head ([D][d + 1], fp32) -> S [D][d] and z [D], set or added
__global__ __launch_bounds__(256) void fwd_export_kernel(const float* __restrict__ X, int64_t head_stride,
                                                         float* __restrict__ S, float* __restrict__ z, int heads,
                                                         int D, int d, int accumulate) {
  const int64_t per = (int64_t)D * (d + 1);
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < (int64_t)heads * per;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t h = i / per, rest = i - h * per;
    const int f = (int)(rest / (d + 1)), c = (int)(rest - (int64_t)f * (d + 1));
    const float v = X[h * head_stride + rest];
    float* dst = c < d ? &S[(h * D + f) * d + c] : &z[h * D + f];
    *dst = accumulate ? *dst + v : v;
  }
}

// ---------------------------------------------------------------------------
// [W | b] in fp32, per parameter set: the projection u = [x | 1] [W | b]^T
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void bwd_packw_kernel(const T* __restrict__ W, const float* __restrict__ b,
                                                        float* __restrict__ Wx, int rows, int d) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * (d + 1)) return;
  const int r = i / (d + 1), c = i - r * (d + 1);
  Wx[i] = c < d ? (float)W[(size_t)r * d + c] : b[r];
}

// ---------------------------------------------------------------------------
// feature-map backward: one thread per (row, projection).  From u and dphi of the
// row, on u's segment: y'_l = s'_l u + t'_l (the table's slope and intercept, scaled by
// 1/sqrt(M)), g_l = dphi_l where the output ReLU passes (y' > 0, or always without
// it), du = sum_l g_l s'_l, and into the (segment, channel) moments dy_l = g_l / sqrt(M)
// and dy_l u (LDS, one copy per workgroup, written out as partials).
// ---------------------------------------------------------------------------
template <int L>
__global__ __launch_bounds__(256) void bwd_phi_kernel(BwdPhi a) {
  constexpr int NSEG = nseg_cap(L, kFmSegBytes);
  __shared__ PwlLds<L, NSEG> tab;
  // per (channel, segment): sum dy and sum dy u, channel-major so that the lanes of
  // one atomic instruction (one channel, random segments) spread over the banks
  __shared__ float m0[L][NSEG], m1[L][NSEG];
  const int set = blockIdx.y, tid = threadIdx.x;
  const int M = a.M, D = M * L;
  pwl_load(tab, a.tables + (size_t)set * kTableBytes);
  for (int i = tid; i < NSEG * L; i += blockDim.x) {
    m0[i / NSEG][i % NSEG] = 0.0f;
    m1[i / NSEG][i % NSEG] = 0.0f;
  }
  __syncthreads();
  const int steps = __builtin_amdgcn_readfirstlane(tab.steps);
  const float floor = tab.floor;
  const float rsm = 1.0f / sqrtf((float)M);
  const int64_t heads_in_set = a.per_head ? a.heads / a.H : a.heads;
  const int64_t per_side = heads_in_set * a.n * M;  // elements (row, projection) of one side
  const int64_t total = 2 * per_side;
  // NB elements per thread and round, their loads issued before any is used
  constexpr int NB = 4;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e0 = blockIdx.x * (int64_t)blockDim.x + tid; e0 < total; e0 += NB * stride) {
    float u[NB], gv[NB][L];
    int64_t ui[NB];
    int side[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int64_t e = min(e0 + b * stride, total - 1);  // (clamped: loads stay in range)
      side[b] = e >= per_side;
      const int64_t el = e - side[b] * per_side;
      const int64_t hs = el / (a.n * M);
      const int64_t rest = el - hs * a.n * M;  // t M + i
      const int i = (int)(rest % M);
      const int64_t head = a.per_head ? hs * a.H + set : hs;
      ui[b] = head * a.n * M + rest;
      u[b] = (side[b] ? a.uk : a.uq)[ui[b]];
      const float* g = (side[b] ? a.dphik : a.dphiq) + head * a.n * D + (rest - i) / M * D + (int64_t)i * L;
      if constexpr (L % 4 == 0) {
#pragma unroll
        for (int q = 0; q < L / 4; ++q) {
          const float4 v = reinterpret_cast<const float4*>(g)[q];
          gv[b][4 * q] = v.x; gv[b][4 * q + 1] = v.y; gv[b][4 * q + 2] = v.z; gv[b][4 * q + 3] = v.w;
        }
      } else {
#pragma unroll
        for (int l = 0; l < L; ++l) gv[b][l] = g[l];
      }
    }
    int sg[NB];
    pwl_search(tab, steps, u, sg);
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (e0 + b * stride >= total) break;
      const float2* row = reinterpret_cast<const float2*>(seg_ptr(tab, sg[b]));
      float du = 0.0f;
#pragma unroll
      for (int l = 0; l < L; ++l) {
        const float2 st = row[l];
        const float gl = fmaf(st.x, u[b], st.y) > floor ? gv[b][l] : 0.0f;  // floor: 0 (output ReLU) or -inf
        du = fmaf(gl, st.x, du);
        if (gl != 0.0f) {  // (channels cut by the output ReLU add nothing)
          const float dy = gl * rsm;
          atomicAdd(&m0[l][sg[b]], dy);
          atomicAdd(&m1[l][sg[b]], dy * u[b]);
        }
      }
      (side[b] ? a.duk : a.duq)[ui[b]] = du;
    }
  }
  __syncthreads();
  float* part = a.partial + ((size_t)set * gridDim.x + blockIdx.x) * a.part_floats;
  const int nm = tab.zero_seg * L;  // real segments x channels
  for (int i = tid; i < nm; i += blockDim.x) {  // partials as [segment][channel][2]
    part[2 * i] = m0[i % L][i / L];
    part[2 * i + 1] = m1[i % L][i / L];
  }
}

// ---------------------------------------------------------------------------
// [dW | db] per parameter set from the per-(batch, head) products dU^T [X | 1]
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void bwd_dw_kernel(const float* __restrict__ dwh, float* __restrict__ dW,
                                                     float* __restrict__ db, int B, int H, int M, int d,
                                                     int per_head) {
  const int E = d + 1;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;  // (set, i, c)
  const int sets = per_head ? H : 1;
  if (idx >= sets * M * E) return;
  const int set = idx / (M * E), rest = idx - set * M * E;
  double s = 0.0;
  for (int bb = 0; bb < B; ++bb)
    for (int hh = per_head ? set : 0; hh < (per_head ? set + 1 : H); ++hh)
      s += (double)dwh[((size_t)bb * H + hh) * M * E + rest];
  const int i = rest / E, c = rest - i * E;
  if (c < d) dW[((size_t)set * M + i) * d + c] = (float)s;
  else db[(size_t)set * M + i] = (float)s;
}

// dX rows [rows][d + 1] (fp32, the last column unused) -> [rows][d] in the call's dtype
template <typename T>
__global__ __launch_bounds__(256) void bwd_cols_kernel(const float* __restrict__ src, T* __restrict__ dst, int64_t rows,
                                                       int d) {
  const int64_t n = rows * d;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / d;
    dst[i] = (T)src[i + r];  // row r starts at r (d + 1)
  }
}

// ---------------------------------------------------------------------------
// partials summed over workgroups (fp64), per parameter set
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void bwd_reduce_kernel(const float* __restrict__ partial, double* __restrict__ sum,
                                                         int groups, int part_floats, int used) {
  const int set = blockIdx.y;
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= used) return;
  const float* p = partial + (size_t)set * groups * part_floats + e;
  double s = 0.0;
  for (int g = 0; g < groups; ++g) s += (double)p[(size_t)g * part_floats];
  sum[(size_t)set * part_floats + e] = s;
}

// ---------------------------------------------------------------------------
// parameter gradients from the reduced sums
// ---------------------------------------------------------------------------

// exclusive prefix sums over segments of the moments of one channel: one workgroup
// per (channel, parameter set), a thread per segment, fp64
__global__ __launch_bounds__(1024) void bwd_prefix_kernel(const double* __restrict__ sum, double* __restrict__ pre,
                                                          const uint8_t* tables, int M, int d, int L, int part_floats,
                                                          int nseg_cap) {
  __shared__ double wtot[2][16];
  const int l = blockIdx.x, set = blockIdx.y, tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
  const PwlHeader hd = *reinterpret_cast<const PwlHeader*>(tables + (size_t)set * kTableBytes + kTabHeader);
  const int nseg = min(max(hd.nbp, 0) + 1, nseg_cap);
  const double* mom = sum + (size_t)set * part_floats;  // [nseg][L][2]
  double* out = pre + ((size_t)set * L + l) * (nseg_cap + 1) * 2;
  double run0 = 0.0, run1 = 0.0;  // the sums of the previous 1024-segment blocks
  for (int j0 = 0; j0 <= nseg; j0 += 1024) {
    const int j = j0 + tid;
    const double v0 = j < nseg ? mom[((size_t)j * L + l) * 2] : 0.0;
    const double v1 = j < nseg ? mom[((size_t)j * L + l) * 2 + 1] : 0.0;
    double i0 = v0, i1 = v1;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const double u0 = __shfl_up(i0, o, kWave), u1 = __shfl_up(i1, o, kWave);
      if (lane >= o) {
        i0 += u0;
        i1 += u1;
      }
    }
    if (lane == kWave - 1) {
      wtot[0][wave] = i0;
      wtot[1][wave] = i1;
    }
    __syncthreads();
    double b0 = run0, b1 = run1;
    for (int w = 0; w < wave; ++w) {
      b0 += wtot[0][w];
      b1 += wtot[1][w];
    }
    if (j <= nseg) {
      out[2 * j] = b0 + i0 - v0;
      out[2 * j + 1] = b1 + i1 - v1;
    }
    double t0 = 0.0, t1 = 0.0;
    for (int w = 0; w < 16; ++w) {
      t0 += wtot[0][w];
      t1 += wtot[1][w];
    }
    run0 += t0;
    run1 += t1;
    __syncthreads();
  }
}

__device__ __forceinline__ uint32_t ordered_key(float x) {
  const uint32_t b = __float_as_uint(x);
  return (b >> 31) ? ~b : (b | 0x80000000u);
}

__global__ __launch_bounds__(256) void bwd_mlp_kernel(BwdMlp a) {
  __shared__ float keys[kKeyCap];
  const int set = blockIdx.x, tid = threadIdx.x;
  const uint8_t* tab = a.tables + (size_t)set * kTableBytes;
  const PwlHeader hd = *reinterpret_cast<const PwlHeader*>(tab + kTabHeader);
  const int nbp = min(max(hd.nbp, 0), a.nseg_cap - 1);
  const int nseg = nbp + 1;
  const float* gkeys = reinterpret_cast<const float*>(tab + kTabKeys);
  for (int i = tid; i < nbp; i += blockDim.x) keys[i] = gkeys[i];
  const int L = a.L, hidden = a.hidden, C1 = a.C1;
  __syncthreads();
  const float* A = a.fc1_w + (size_t)set * C1 * hidden;
  const float* Cc = a.fc1_b + (size_t)set * C1 * hidden;
  const float* F = a.fc2_w + (size_t)set * L * hidden;
  const double* preset = a.pre + (size_t)set * L * (a.nseg_cap + 1) * 2;
  // sums of the moments of channel l over the segments where a unit (a, c) is on
  auto on_sums = [&](int l, float ak, float ck, double& m0, double& m1) {
    const double* P = preset + (size_t)l * (a.nseg_cap + 1) * 2;
    const float q = (float)(-(double)ck / (double)ak);
    if (ak != 0.0f && isfinite(q)) {
      // its rank: the number of keys below the breakpoint (for equal keys any of
      // them: the segments between equal keys are empty)
      const uint32_t kb = ordered_key(q == 0.0f ? 0.0f : q);
      int lo = 0, hi = nbp;
      while (lo < hi) {
        const int mid = (lo + hi) / 2;
        if (ordered_key(keys[mid]) < kb) lo = mid + 1;
        else hi = mid;
      }
      if (ak > 0.0f) {  // on above the breakpoint: segments j > rank
        m0 = P[2 * nseg] - P[2 * (lo + 1)];
        m1 = P[2 * nseg + 1] - P[2 * (lo + 1) + 1];
      } else {          // on below it: segments j <= rank
        m0 = P[2 * (lo + 1)];
        m1 = P[2 * (lo + 1) + 1];
      }
    } else if (ck > 0.0f) {  // constant and on
      m0 = P[2 * nseg];
      m1 = P[2 * nseg + 1];
    } else {
      m0 = m1 = 0.0;
    }
  };
  for (int idx = tid; idx < L * hidden; idx += blockDim.x) {
    const int l = idx / hidden, k = idx - l * hidden;
    const int u = (C1 == 1 ? 0 : l) * hidden + k;
    double m0, m1;
    on_sums(l, A[u], Cc[u], m0, m1);
    a.dfc2_w[(size_t)set * L * hidden + idx] = (float)((double)A[u] * m1 + (double)Cc[u] * m0);
  }
  for (int l = tid; l < L; l += blockDim.x)
    a.dfc2_b[(size_t)set * L + l] = (float)preset[((size_t)l * (a.nseg_cap + 1) + nseg) * 2];
  for (int u = tid; u < C1 * hidden; u += blockDim.x) {
    const int k = u % hidden;
    const int l0 = C1 == 1 ? 0 : u / hidden, l1 = C1 == 1 ? L : u / hidden + 1;
    double g1 = 0.0, g0 = 0.0;
    for (int l = l0; l < l1; ++l) {
      double m0, m1;
      on_sums(l, A[u], Cc[u], m0, m1);
      const double f = (double)F[l * hidden + k];
      g1 += f * m1;
      g0 += f * m0;
    }
    a.dfc1_w[(size_t)set * C1 * hidden + u] = (float)g1;
    a.dfc1_b[(size_t)set * C1 * hidden + u] = (float)g0;
  }
}

}  // namespace

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
hipError_t launch_bwd_pack(Dt dt, const void* V, float* Vx, int64_t rows, int d, hipStream_t s) {
  const int64_t total = rows * (d + 1);
  const dim3 grid((unsigned)std::min<int64_t>((total + 255) / 256, 65536)), block(256);
  if (dt == Dt::BF16) hipLaunchKernelGGL(bwd_pack_kernel<__bf16>, grid, block, 0, s, (const __bf16*)V, Vx, rows, d);
  else hipLaunchKernelGGL(bwd_pack_kernel<float>, grid, block, 0, s, (const float*)V, Vx, rows, d);
  return hipGetLastError();
}

hipError_t launch_bwd_convert(Dt dt, const float* src, void* dst, int64_t n, hipStream_t s) {
  const dim3 grid((unsigned)std::min<int64_t>((n + 255) / 256, 65536)), block(256);
  if (dt == Dt::BF16) hipLaunchKernelGGL(bwd_convert_kernel<__bf16>, grid, block, 0, s, src, (__bf16*)dst, n);
  else hipLaunchKernelGGL(bwd_convert_kernel<float>, grid, block, 0, s, src, (float*)dst, n);
  return hipGetLastError();
}

hipError_t launch_bwd_gemm(const BwdGemm& g, hipStream_t s) {
  // at most 65535 (head, chunk) batches per launch: whole heads per slice
  const int per = std::max(1, 65535 / std::max(1, g.chunks));
  for (int h0 = 0; h0 < g.heads; h0 += per) {
    BwdGemm q = g;
    q.heads = std::min(per, g.heads - h0);
    q.A = g.A + h0 * g.sAh;
    q.B = g.B + h0 * g.sBh;
    q.C = g.C + h0 * g.sCh;
    const dim3 grid((unsigned)((g.N + kGT - 1) / kGT), (unsigned)((g.M + kGT - 1) / kGT),
                    (unsigned)(q.heads * g.chunks));
    hipLaunchKernelGGL(bwd_gemm_kernel, grid, dim3(256), 0, s, q);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_bwd_scan(float* X, int heads, int chunks, int64_t elems, int mode, hipStream_t s) {
  for (int h0 = 0; h0 < heads; h0 += 65535) {  // at most 65535 heads per launch
    const int hn = std::min(65535, heads - h0);
    const dim3 grid((unsigned)((elems + 255) / 256), (unsigned)hn);
    hipLaunchKernelGGL(bwd_scan_kernel, grid, dim3(256), 0, s, X + (int64_t)h0 * chunks * elems, hn, chunks, elems,
                       mode);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_bwd_g(Dt dt, float* Y, const void* dO, int64_t rows, int d, float eps, hipStream_t s) {
  const dim3 grid((unsigned)((rows + 3) / 4)), block(256);
  if (dt == Dt::BF16) hipLaunchKernelGGL(bwd_g_kernel<__bf16>, grid, block, 0, s, Y, (const __bf16*)dO, rows, d, eps);
  else hipLaunchKernelGGL(bwd_g_kernel<float>, grid, block, 0, s, Y, (const float*)dO, rows, d, eps);
  return hipGetLastError();
}

int bwd_phi_groups(int64_t rows_per_set) {
  return (int)std::max<int64_t>(1, std::min<int64_t>((rows_per_set + 1023) / 1024, 512));
}

bool bwd_supported(int d, int L, int M) {
  const bool lok = L == 1 || L == 2 || L == 4 || L == 8 || L == 16;
  return lok && M >= 1 && M <= 256 && M * L <= 256 && d >= 1 && d <= 128;
}

size_t bwd_part_floats(int, int L, int) { return 2 * (size_t)nseg_cap(L, kFmSegBytes) * L; }

hipError_t launch_bwd_packw(Dt dt, const void* W, const float* b, float* Wx, int rows, int d, hipStream_t s) {
  const dim3 grid((unsigned)((rows * (d + 1) + 255) / 256)), block(256);
  if (dt == Dt::BF16) hipLaunchKernelGGL(bwd_packw_kernel<__bf16>, grid, block, 0, s, (const __bf16*)W, b, Wx, rows, d);
  else hipLaunchKernelGGL(bwd_packw_kernel<float>, grid, block, 0, s, (const float*)W, b, Wx, rows, d);
  return hipGetLastError();
}

hipError_t launch_bwd_phi(int L, const BwdPhi& a, int groups, int sets, hipStream_t s) {
  const dim3 grid((unsigned)groups, (unsigned)sets);
  switch (L) {
    case 1: hipLaunchKernelGGL(bwd_phi_kernel<1>, grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL(bwd_phi_kernel<2>, grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL(bwd_phi_kernel<4>, grid, dim3(256), 0, s, a); break;
    case 8: hipLaunchKernelGGL(bwd_phi_kernel<8>, grid, dim3(256), 0, s, a); break;
    case 16: hipLaunchKernelGGL(bwd_phi_kernel<16>, grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_bwd_dw(const float* dwh, float* dW, float* db, int B, int H, int M, int d, int per_head,
                         hipStream_t s) {
  const int total = (per_head ? H : 1) * M * (d + 1);
  hipLaunchKernelGGL(bwd_dw_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, dwh, dW, db, B, H, M, d,
                     per_head);
  return hipGetLastError();
}

hipError_t launch_bwd_cols(Dt dt, const float* src, void* dst, int64_t rows, int d, hipStream_t s) {
  const dim3 grid((unsigned)std::min<int64_t>((rows * d + 255) / 256, 65536)), block(256);
  if (dt == Dt::BF16) hipLaunchKernelGGL(bwd_cols_kernel<__bf16>, grid, block, 0, s, src, (__bf16*)dst, rows, d);
  else hipLaunchKernelGGL(bwd_cols_kernel<float>, grid, block, 0, s, src, (float*)dst, rows, d);
  return hipGetLastError();
}

hipError_t launch_bwd_reduce(const float* partial, double* sum, int groups, int part_floats, int used, int sets,
                             hipStream_t s) {
  const dim3 grid((unsigned)((used + 255) / 256), (unsigned)sets);
  hipLaunchKernelGGL(bwd_reduce_kernel, grid, dim3(256), 0, s, partial, sum, groups, part_floats, used);
  return hipGetLastError();
}

hipError_t launch_bwd_prefix(const double* sum, double* pre, const uint8_t* tables, int M, int d, int L,
                             int part_floats, int nseg_cap_, int sets, hipStream_t s) {
  hipLaunchKernelGGL(bwd_prefix_kernel, dim3((unsigned)L, (unsigned)sets), dim3(1024), 0, s, sum, pre, tables, M, d, L,
                     part_floats, nseg_cap_);
  return hipGetLastError();
}

hipError_t launch_bwd_mlp(const BwdMlp& a, int sets, hipStream_t s) {
  hipLaunchKernelGGL(bwd_mlp_kernel, dim3((unsigned)sets), dim3(256), 0, s, a);
  return hipGetLastError();
}

int bwd_nseg_cap(int L) { return nseg_cap(L, kFmSegBytes); }

hipError_t launch_fwd_out(Dt dt, const float* Y, void* out, int64_t rows, int d, float eps, hipStream_t s) {
  const dim3 grid((unsigned)((rows + 3) / 4)), block(256);
  if (dt == Dt::BF16) hipLaunchKernelGGL(fwd_out_kernel<__bf16>, grid, block, 0, s, Y, (__bf16*)out, rows, d, eps);
  else hipLaunchKernelGGL(fwd_out_kernel<float>, grid, block, 0, s, Y, (float*)out, rows, d, eps);
  return hipGetLastError();
}

hipError_t launch_fwd_export(const float* X, int64_t head_stride, float* S, float* z, int heads, int D, int d,
                             int accumulate, hipStream_t s) {
  const int64_t total = (int64_t)heads * D * (d + 1);
  const dim3 grid((unsigned)std::min<int64_t>((total + 255) / 256, 65536)), block(256);
  hipLaunchKernelGGL(fwd_export_kernel, grid, block, 0, s, X, head_stride, S, z, heads, D, d, accumulate);
  return hipGetLastError();
}

}  // namespace luna
