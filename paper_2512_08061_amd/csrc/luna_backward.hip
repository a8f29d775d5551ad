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
// an exact regrouping of the sums.  The non-causal form is the same with one chunk of
// the whole sequence, the total state in place of the prefix and suffix states and no
// intra-chunk terms.
//
// Kernels (all arithmetic in fp32):
//   bwd_pack_kernel     V -> [V | 1] in fp32;
//   bwd_gemm_kernel     batched C (+)= A B over (head, chunk) with strided operands, a
//                       lower-triangular output mask and ragged last chunks;
//   bwd_scan_kernel     exclusive prefix or suffix sums of the per-chunk states;
//   bwd_g_kernel        [num | den - eps] -> G = [dnum | dden];
//   bwd_phi_kernel      dphi -> du (slopes of the piecewise-linear channel functions,
//                       zero where the output ReLU is off) -> dx = du W, with per
//                       workgroup partial dW, db and, per (segment, channel), the
//                       moments sum dy and sum dy u of the channel outputs' gradients;
//   bwd_reduce_kernel   the partials summed over workgroups (fp64);
//   bwd_prefix_kernel   exclusive prefix sums of the moments over segments, per channel;
//   bwd_mlp_kernel      the channel-MLP parameter gradients from the moments: unit k
//                       is on exactly on the segments above (a_k > 0) or below
//                       (a_k < 0) its breakpoint, where h_k = a_k u + c_k, so
//                       dfc2_lk = a_k sum_on dy_l u + c_k sum_on dy_l,
//                       dfc1_(l)k = f_lk sum_on dy_l u, dfc1_b likewise, dfc2_b_l = sum dy_l.
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
// batched strided GEMM, 64 x 64 output tiles, 16-deep k slices through LDS
// ---------------------------------------------------------------------------
constexpr int kGT = 64, kGK = 16;

__global__ __launch_bounds__(256) void bwd_gemm_kernel(BwdGemm g) {
  __shared__ float As[kGK][kGT + 1];
  __shared__ float Bs[kGK][kGT + 1];
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
  const int tid = threadIdx.x;
  const int ti = tid / 16, tj = tid % 16;  // 4 x 4 outputs: rows ti + 16 r, columns tj + 16 q
  float acc[4][4];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[r][q] = 0.0f;
  for (int k0 = 0; k0 < Kv; k0 += kGK) {
#pragma unroll
    for (int e = 0; e < (kGK * kGT) / 256; ++e) {
      const int idx = tid + 256 * e;
      const int kk = idx / kGT, ii = idx % kGT;
      const int k = k0 + kk;
      const int ia = i0 + ii, jb = j0 + ii;
      As[kk][ii] = (k < Kv && ia < Mv) ? A[ia * g.sAi + k * g.sAk] : 0.0f;
      Bs[kk][ii] = (k < Kv && jb < Nv) ? B[k * g.sBk + jb * g.sBj] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kGK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) a[r] = As[kk][ti + 16 * r];
#pragma unroll
      for (int q = 0; q < 4; ++q) b[q] = Bs[kk][tj + 16 * q];
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[r][q] = fmaf(a[r], b[q], acc[r][q]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int i = i0 + ti + 16 * r;
    if (i >= Mv) continue;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int j = j0 + tj + 16 * q;
      if (j >= Nv) continue;
      float v = (g.lower && j > i) ? 0.0f : acc[r][q];
      float* p = C + i * g.sCi + j * g.sCj;
      if (g.accumulate) v += *p;
      *p = v;
    }
  }
}

// ---------------------------------------------------------------------------
// exclusive prefix (forward) or suffix (backward) sums over chunks, in place
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void bwd_scan_kernel(float* X, int heads, int chunks, int64_t elems, int suffix) {
  const int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int h = blockIdx.y;
  if (e >= elems || h >= heads) return;
  float* base = X + (int64_t)h * chunks * elems + e;
  float run = 0.0f;
  for (int i = 0; i < chunks; ++i) {
    const int c = suffix ? chunks - 1 - i : i;
    const float v = base[(int64_t)c * elems];
    base[(int64_t)c * elems] = run;
    run += v;
  }
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
// feature-map backward
// ---------------------------------------------------------------------------
constexpr int kPhiRows = 32;  // rows per tile
constexpr int kPhiMaxM = 64, kPhiMaxD = 128;

template <typename T, int L>
__global__ __launch_bounds__(256) void bwd_phi_kernel(BwdPhi a) {
  constexpr int NSEG = nseg_cap(L, kFmSegBytes);
  __shared__ PwlLds<L, NSEG> tab;
  __shared__ float Ws[kPhiMaxM * kPhiMaxD];
  __shared__ float xs[kPhiRows][kPhiMaxD + 1];
  __shared__ float dus[kPhiRows][kPhiMaxM + 1];
  __shared__ float mom[NSEG * L][2];  // per (segment, channel): sum dy, sum dy u

  const int set = blockIdx.y;  // parameter set; its workgroups share the tiles of its heads
  const int tid = threadIdx.x;
  const int M = a.M, d = a.d, D = M * L;
  const float* bias = a.b + (size_t)set * M;
  const T* W = reinterpret_cast<const T*>(a.W) + (size_t)set * M * d;
  pwl_load(tab, a.tables + (size_t)set * kTableBytes);
  for (int i = tid; i < M * d; i += blockDim.x) Ws[i] = (float)W[i];
  for (int i = tid; i < NSEG * L; i += blockDim.x) mom[i][0] = mom[i][1] = 0.0f;
  __syncthreads();
  const int steps = __builtin_amdgcn_readfirstlane(tab.steps);
  const float floor = tab.floor;
  const float rsm = 1.0f / sqrtf((float)M);

  // this thread's share of the partial dW (rows i, columns c: entries tid, tid + 256, ...)
  constexpr int kMaxW = kPhiMaxM * kPhiMaxD / 256;
  float dw[kMaxW];
#pragma unroll
  for (int e = 0; e < kMaxW; ++e) dw[e] = 0.0f;
  float dbias = 0.0f;  // thread i < M: partial db_i

  // tiles: rows of the heads of this parameter set, Q rows then K rows
  const int64_t heads_in_set = a.per_head ? a.heads / a.H : a.heads;
  const int64_t tiles_per_head = (a.n + kPhiRows - 1) / kPhiRows;
  const int64_t tiles = 2 * heads_in_set * tiles_per_head;
  const int r = tid / 8, pg = tid % 8;  // row of the tile, projection group (i = pg, pg + 8, ...)
  for (int64_t it = blockIdx.x; it < tiles; it += gridDim.x) {
    const int side = (int)(it / (heads_in_set * tiles_per_head));  // 0: Q rows, 1: K rows
    const int64_t rest = it - side * heads_in_set * tiles_per_head;
    const int64_t hs = rest / tiles_per_head;
    const int64_t t0 = (rest - hs * tiles_per_head) * kPhiRows;
    const int64_t head = a.per_head ? hs * a.H + set : hs;
    const T* X = reinterpret_cast<const T*>(side ? a.K : a.Q) + head * a.n * d;
    const float* dphi = (side ? a.dphik : a.dphiq) + head * a.n * D;
    T* dX = reinterpret_cast<T*>(side ? a.dK : a.dQ) + head * a.n * d;
    const int rows = (int)min((int64_t)kPhiRows, a.n - t0);
    __syncthreads();  // the previous tile's xs and dus are no longer read
    for (int i = tid; i < kPhiRows * d; i += blockDim.x) {
      const int rr = i / d, cc = i - rr * d;
      xs[rr][cc] = rr < rows ? (float)X[(t0 + rr) * d + cc] : 0.0f;
    }
    __syncthreads();
    if (r < rows) {
      const float* g = dphi + (t0 + r) * D;
      for (int i = pg; i < M; i += 8) {
        float u = bias[i];
        for (int cc = 0; cc < d; ++cc) u = fmaf(Ws[i * d + cc], xs[r][cc], u);
        float uu[1] = {u};
        int sg[1];
        pwl_search(tab, steps, uu, sg);
        const float4* row = reinterpret_cast<const float4*>(seg_ptr(tab, sg[0]));
        float du = 0.0f;
#pragma unroll
        for (int l = 0; l < L; ++l) {
          const float2 st = reinterpret_cast<const float2*>(row)[l];
          const float y = fmaf(st.x, u, st.y);                 // pre-ReLU channel output / sqrt(M)
          const float gl = (y > floor) ? g[i * L + l] : 0.0f;  // floor: 0 (output ReLU) or -inf
          du = fmaf(gl, st.x, du);
          const float dy = gl * rsm;                            // dL / dy_l
          atomicAdd(&mom[sg[0] * L + l][0], dy);
          atomicAdd(&mom[sg[0] * L + l][1], dy * u);
        }
        dus[r][i] = du;
      }
    }
    __syncthreads();
    // dx = du W for the tile's rows; partial dW += du^T x; db += du
    for (int i = tid; i < kPhiRows * d; i += blockDim.x) {
      const int rr = i / d, cc = i - rr * d;
      if (rr < rows) {
        float s = 0.0f;
        for (int p = 0; p < M; ++p) s = fmaf(dus[rr][p], Ws[p * d + cc], s);
        dX[(t0 + rr) * d + cc] = (T)s;
      }
    }
#pragma unroll
    for (int e = 0; e < kMaxW; ++e) {
      const int idx = tid + 256 * e;
      if (idx < M * d) {
        const int i = idx / d, cc = idx - i * d;
        float s = 0.0f;
        for (int rr = 0; rr < rows; ++rr) s = fmaf(dus[rr][i], xs[rr][cc], s);
        dw[e] += s;
      }
    }
    if (tid < M)
      for (int rr = 0; rr < rows; ++rr) dbias += dus[rr][tid];
  }
  __syncthreads();
  // partials of this workgroup
  float* part = a.partial + ((size_t)set * gridDim.x + blockIdx.x) * a.part_floats;
#pragma unroll
  for (int e = 0; e < kMaxW; ++e) {
    const int idx = tid + 256 * e;
    if (idx < M * d) part[idx] = dw[e];
  }
  if (tid < M) part[M * d + tid] = dbias;
  const int nm = tab.zero_seg * L;  // real segments x channels
  for (int i = tid; i < nm; i += blockDim.x) {
    part[M * d + M + 2 * i] = mom[i][0];
    part[M * d + M + 2 * i + 1] = mom[i][1];
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
  const double* mom = sum + (size_t)set * part_floats + (size_t)M * d + M;  // [nseg][L][2]
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
  const double* sum = a.sum + (size_t)set * a.part_floats;
  const int M = a.M, d = a.d, L = a.L, hidden = a.hidden, C1 = a.C1;
  // dW and db straight from the sums
  for (int i = tid; i < M * d; i += blockDim.x) a.dW[(size_t)set * M * d + i] = (float)sum[i];
  for (int i = tid; i < M; i += blockDim.x) a.db[(size_t)set * M + i] = (float)sum[M * d + i];
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

hipError_t launch_bwd_scan(float* X, int heads, int chunks, int64_t elems, int suffix, hipStream_t s) {
  for (int h0 = 0; h0 < heads; h0 += 65535) {  // at most 65535 heads per launch
    const int hn = std::min(65535, heads - h0);
    const dim3 grid((unsigned)((elems + 255) / 256), (unsigned)hn);
    hipLaunchKernelGGL(bwd_scan_kernel, grid, dim3(256), 0, s, X + (int64_t)h0 * chunks * elems, hn, chunks, elems,
                       suffix);
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
  const int64_t tiles = 2 * ((rows_per_set + kPhiRows - 1) / kPhiRows);
  return (int)std::max<int64_t>(1, std::min<int64_t>(tiles, 256));
}

bool bwd_supported(int d, int L, int M) {
  const bool lok = L == 1 || L == 2 || L == 4 || L == 8 || L == 16;
  return lok && M >= 1 && M <= kPhiMaxM && d >= 1 && d <= kPhiMaxD;
}

size_t bwd_part_floats(int d, int L, int M) {
  return (size_t)M * d + M + 2 * (size_t)nseg_cap(L, kFmSegBytes) * L;
}

template <typename T>
static hipError_t phi_dispatch(int L, const BwdPhi& a, dim3 grid, hipStream_t s) {
  switch (L) {
    case 1: hipLaunchKernelGGL((bwd_phi_kernel<T, 1>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((bwd_phi_kernel<T, 2>), grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((bwd_phi_kernel<T, 4>), grid, dim3(256), 0, s, a); break;
    case 8: hipLaunchKernelGGL((bwd_phi_kernel<T, 8>), grid, dim3(256), 0, s, a); break;
    case 16: hipLaunchKernelGGL((bwd_phi_kernel<T, 16>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_bwd_phi(Dt dt, int L, const BwdPhi& a, int groups, int sets, hipStream_t s) {
  const dim3 grid((unsigned)groups, (unsigned)sets);
  return dt == Dt::BF16 ? phi_dispatch<__bf16>(L, a, grid, s) : phi_dispatch<float>(L, a, grid, s);
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

}  // namespace luna
