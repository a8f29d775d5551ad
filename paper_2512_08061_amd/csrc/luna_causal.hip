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
// Work split.  One workgroup owns one (head, part of the sequence).  With fewer heads
// than compute units a call makes two launches, and no workgroup waits for another:
//  - staged (97 to 128 heads): two launches of the scan kernel with explicit chunk
//    ranges per part.  The first scans [0, A) beside a part that only sums the state
//    of [A, A + B), both writing their final states; the second scans [A, A + B) and
//    [A + B, nch) from those states (A = nch / 5, B = 2 nch / 5: a state-only chunk
//    costs about half a scanned one, so both launches are balanced);
//  - otherwise each head is cut at a chunk boundary x near n/2: the state launch (a
//    separate instantiation, ST) sums the state of [0, x) in pieces, one workgroup per
//    (head, piece), and writes them in fp32; the scan launch then runs part 0 over
//    [0, x) from a zero state and part 1 over [x, n) from the sum of the pieces.
// Run over every chunk (key rows past n mapped to the all-zero segment), the state
// launch also gives the state of a whole sequence, which causal_state_export_kernel
// writes in the public layout.
//
// Roles.  Four matrix waves and four map waves, one of each on every SIMD, so that
// each SIMD pairs matrix-core work with vector and table-lookup work.  (With PF, the
// features are given: phi(Q) and phi(K) in bf16, [head][token][FP], written by the
// feature-map kernel, for feature maps whose projections and tables do not fit the map
// waves' registers and LDS, such as one channel per projection with M = 256.  The map
// waves then only copy phi(Q) rows, transpose phi(K) in registers and sum z.)
//  - Map wave b maps rows 16 b .. 16 b + 15 of the next chunk's queries and keys for
//    all projections (the projection on the matrix cores with W fragments and biases
//    in registers, then the piecewise-linear channel functions from the LDS table),
//    stages a share of V, and accumulates z with one-hot matrix-core columns.  phi(Q)
//    is stored token-major and phi(K) feature-major in LDS.
//  - Matrix wave w owns value columns 32 w .. 32 w + 31 and keeps that slice of S (all
//    features) in fp32 accumulators.
// Per chunk c, two barriers:
//   B1: phi(Q_c), phi(K_c), V_c and z_{c-1} are in LDS.
//       matrix: one pass over phi(Q_c) forms the readout S_{c-1}^T phi(Q_c)^T (S taken
//       straight from the accumulators), this wave's P^T blocks and one block of
//       phi(Q_c) z_{c-1}; then the V_c fragments and S += phi(K_c)^T V_c.
//       map: chunk c + 1's projections and table searches; phi(Q_{c+1}) evaluated.
//   B2: P and the den parts are in LDS; chunk c's tiles are no longer read.
//       matrix: num^T += V^T P^T, the division and the store.
//       map: phi(Q_{c+1}) to LDS, phi(K_{c+1}) evaluated and stored, z and V_{c+1}.
//
// The loop is bound by LDS instructions and their latency, so its tiles are laid out for
// addressing without arithmetic: rows are padded by 16 bytes instead of swizzled
// (16 consecutive rows then start on 16 distinct 16-byte bank slots), so that every
// operand a lane reads or writes is one base register plus a constant the LDS
// instruction carries.  Features are numbered so that the phi(K)^T rows one map wave
// writes, and each 16-feature block of S, are 16 consecutive rows.  Q, K, V and the
// output go through range-checked buffer instructions: rows past the end read as 0
// and are not written, with no per-lane tests.
#include "luna_device.hpp"
#include "luna_kernels.hpp"

#include <type_traits>

namespace luna {

template <typename T, int DH, int L, int MB, bool PF = false>
struct CsCfg {
  static constexpr int NCB = DH / 16;             // 16-column blocks of the value width
  static constexpr int NMW = NCB < 4 ? NCB : 4;   // matrix waves that own value columns
  static constexpr int CBW = NCB / NMW;           // 16-column blocks per matrix wave
  static constexpr int NMS = 4;                   // matrix-wave slots (the extra ones idle)
  static constexpr int NT = 512;                  // four matrix and four map waves
  static constexpr int KS = DH / 32;              // 32-wide k-steps of the projection
  static constexpr int FP = 16 * MB * L;          // features, projections padded to 16
  static constexpr int NF = FP / 32;              // 32-feature k-fragments
  static constexpr int RB = FP / 16;              // 16-feature row blocks of S
  static constexpr int SZ = (int)sizeof(T);
  static constexpr int VE = 16 / SZ;              // elements per 16-byte chunk
  static constexpr int SQ = FP * SZ + 16;         // phi(Q) row stride (bytes)
  static constexpr int SK = 64 * SZ + 16;         // phi(K)^T row stride
  static constexpr int SP = 64 * SZ + 16;         // P row stride
  static constexpr int VPT = 64 * DH / VE / 256;  // 16-byte V chunks per map-wave thread
  static constexpr int NSEG = nseg_cap(L, kAttnSegBytes);
  // one state piece: the matrix waves' S slices (lane-major accumulator tiles), then z
  static constexpr int SF = NMW * CBW * RB * kWave * 4;
  static constexpr int STATE = (SF + FP + 63) / 64 * 64;
  // bf16: fp16 coefficient rows and keys in 4-key groups; fp32: fp32 rows and plain keys;
  // features given: no table
  struct NoTab {};
  using Tab = typename std::conditional<
      PF, NoTab, typename std::conditional<SZ == 2, PwlLdsN<half2_t, L, NSEG>, PwlLds<L, NSEG>>::type>::type;
  static constexpr int WMB = PF ? 1 : MB;  // W fragment blocks held in LDS
  static_assert(NCB == 2 || NCB == 4 || NCB == 8, "d must be 32, 64 or 128");
  static_assert(FP % 32 == 0 && (PF || (L % 2 == 0 && (SZ == 4 || L % 4 == 0))),
                "features must fill 32-wide fragments");
  static_assert(!PF || (SZ == 2 && L == 1 && (FP == 128 || FP == 256)),
                "given features: bf16, 128 or 256 of them");
  static_assert(VPT * 256 * VE == 64 * DH, "V chunks must split evenly over the map threads");
};

// The small arrays that are addressed with constant indices come first, and the
// table's keys right after them: below 64 KiB their addresses fit the 16-bit
// offset of an LDS instruction, so that such accesses need no address register.
template <typename T, int DH, int L, int MB, bool PF>
struct CsLds {
  using C = CsCfg<T, DH, L, MB, PF>;
  alignas(16) float denp[4][64];           // row sums of P per key block
  alignas(16) float deni[64];              // phi(Q_c) z_{c-1}
  alignas(16) float zp[4][C::FP];          // z_c over each 16-row block of keys
  alignas(16) T zs[2][C::FP];              // z_c, summed, by chunk parity
  float bias[16 * MB];                     // projection biases, 0 for padded projections
  typename C::Tab tab;  // search keys, bucket windows, coefficient rows
  alignas(16) T wfr[C::WMB][C::KS][kWave][8];  // W fragments (A of u^T = W X^T, B of u = X W^T)
  alignas(16) char pm[64 * C::SP];         // P, query-major (blocks above the diagonal stay 0)
  alignas(16) char phq[64 * C::SQ];        // phi(Q_c), token-major, feature f at position f
  alignas(16) char phk[C::FP * C::SK];     // phi(K_c)^T, feature f in row krow(f)
  alignas(16) T vt[64 * DH];               // V_c, token-major (swizzled)
};

// Feature index of projection p and channel l (MB projection blocks of 16).  Bits
// 0-1 and 3-4 hold the projection's place in its block, bit 2 and bits 5.. the
// block and channel, so that krow (below) puts projection block m, channel l in
// rows 16 (m + MB l) .. 16 (m + MB l) + 15.
template <int MB>
__device__ __forceinline__ constexpr int feat(int p, int l) {
  const int pr = p & 15, c = (p >> 4) + MB * l;
  return (pr & 3) | ((c & 1) << 2) | ((pr >> 2) << 3) | ((c >> 1) << 5);
}
// Row of phi(K)^T (and of S) holding feature f: bits 3-4 of f move to 2-3 and bit 2
// to 4.  Row block b of S (rows 16 b .. 16 b + 15) then holds, in its accumulator
// tile row 4 g + jj, feature 32 (b / 2) + 8 g + 4 (b % 2) + jj: tiles 2 kf and
// 2 kf + 1 together are the k-fragment kf of S^T (slot e of lane group g = feature
// 32 kf + 8 g + e) exactly as they stand.
__device__ __forceinline__ constexpr int krow(int f) {
  return (f & ~31) | (f & 3) | ((f >> 1) & 12) | ((f << 2) & 16);
}
// The feature held in row rho (the inverse of krow).
__device__ __forceinline__ constexpr int krow_inv(int rho) {
  return (rho & ~31) | (rho & 3) | ((rho << 1) & 24) | ((rho >> 2) & 4);
}

// V: transpose reads of four (and eight) consecutive rows.
template <int CPR>
__device__ __forceinline__ int swz_v(int row, int cg) {
  const int h = (row & 3) ^ ((row >> 2) & 1) ^ ((row >> 3) & 1);
  return cg ^ ((2 * h) & (CPR - 1));
}

typedef __attribute__((ext_vector_type(4))) unsigned u32x4;

// 8 consecutive elements at LDS byte address p (16 B for bf16, 32 B for fp32)
__device__ __forceinline__ void lds8(Frag<__bf16>& f, const char* p) {
  f.v = *reinterpret_cast<const bf16x8*>(p);
}
__device__ __forceinline__ void lds8(Frag<float>& f, const char* p) {
  const float4 lo = reinterpret_cast<const float4*>(p)[0];
  const float4 hi = reinterpret_cast<const float4*>(p)[1];
  f.v[0] = lo.x; f.v[1] = lo.y; f.v[2] = lo.z; f.v[3] = lo.w;
  f.v[4] = hi.x; f.v[5] = hi.y; f.v[6] = hi.z; f.v[7] = hi.w;
}
// Slots e0 .. e0 + 3 of a k-fragment from four rows (stride bytes apart) of a
// row-major LDS tile, column = this lane's index in its group of 16.  bf16 uses the
// gfx950 transpose read, for which `p` is the address of columns 4 (i % 4) .. of row
// i / 4 (i = lane % 16); fp32 reads its four elements directly, `p` being the
// address of column i of the first row.
__device__ __forceinline__ void load_tr4_rows(Frag<__bf16>& f, int e0, const char* p, int) {
  typedef __attribute__((ext_vector_type(4))) short i16x4;
  const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4*)(__attribute__((address_space(3))) void*)(p));
  const bf16x4 b = __builtin_bit_cast(bf16x4, v);
  f.v[e0 + 0] = b[0]; f.v[e0 + 1] = b[1]; f.v[e0 + 2] = b[2]; f.v[e0 + 3] = b[3];
}
__device__ __forceinline__ void load_tr4_rows(Frag<float>& f, int e0, const char* p, int stride) {
#pragma unroll
  for (int e = 0; e < 4; ++e) f.v[e0 + e] = *reinterpret_cast<const float*>(p + e * stride);
}

// x plus the x of lane l ^ 16 (and l ^ 32).  A permlane swap of a value with itself
// leaves every lane its own value in one result and its partner's in the other.
__device__ __forceinline__ float sum_xor16(float x) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}
__device__ __forceinline__ float sum_xor32(float x) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}

// Four values of one channel (one per projection or token j = 0..3) in the element
// type: written to LDS as one 8-byte (bf16) or 16-byte (fp32) store.
template <typename T>
struct Pack4;
template <>
struct Pack4<__bf16> {
  bf16x4 v;
  __device__ __forceinline__ void set2(int j, float a, float b) {
    typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
    const bf16x2 p = {(__bf16)a, (__bf16)b};
    v[j] = p[0];
    v[j + 1] = p[1];
  }
  __device__ __forceinline__ void store(char* p) const { *reinterpret_cast<bf16x4*>(p) = v; }
  __device__ __forceinline__ void to_frag(Frag<__bf16>& f, int e0) const {
    f.v[e0] = v[0]; f.v[e0 + 1] = v[1]; f.v[e0 + 2] = v[2]; f.v[e0 + 3] = v[3];
  }
};
template <>
struct Pack4<float> {
  float4 v;
  __device__ __forceinline__ void set2(int j, float a, float b) {
    if (j == 0) { v.x = a; v.y = b; }
    else { v.z = a; v.w = b; }
  }
  __device__ __forceinline__ void store(char* p) const { *reinterpret_cast<float4*>(p) = v; }
  __device__ __forceinline__ void to_frag(Frag<float>& f, int e0) const {
    f.v[e0] = v.x; f.v[e0 + 1] = v.y; f.v[e0 + 2] = v.z; f.v[e0 + 3] = v.w;
  }
};

// ST: the state launch (state-only chunks, S and z dumped); otherwise a scan launch.
// PF: the features are given (a.phiq, a.phik); L = 1 and MB = FP / 16.
template <typename T, int DH, int L, int MB, bool ST, bool PF>
__global__ __launch_bounds__(512, 1) void causal_kernel(CausalArgs a) {
  using C = CsCfg<T, DH, L, MB, PF>;
  constexpr int KS = C::KS, FP = C::FP, NF = C::NF, RB = C::RB, VE = C::VE, NMW = C::NMW, NMS = C::NMS;
  constexpr int CBW = C::CBW, SZ = C::SZ, SQ = C::SQ, SK = C::SK, SP = C::SP, CPV = DH / VE;
  constexpr bool kF16 = sizeof(T) == 2;  // fp16 coefficient rows for bf16 data
  __shared__ CsLds<T, DH, L, MB, PF> sm;

  // state launch: one workgroup per (head, piece of the first `split` tokens); scan
  // launch: one per (head, part)
  constexpr bool state_run = ST;
  const int per_head = state_run ? a.pieces : a.parts;
  const int head = blockIdx.x / per_head;
  const int part = blockIdx.x - head * per_head;
  const int hset = a.phi.per_head ? head % a.H : 0;
  if constexpr (!PF) pwl_load(sm.tab, a.phi.tables + (size_t)hset * kTableBytes);

  const int tid = threadIdx.x;
  const int wave = wave_id();
  const int lane = tid % kWave, g = lane / 16, r = lane % 16;
  const int M = a.phi.M;
  const int n = a.n;
  const size_t hoff = (size_t)head * n * DH;
  const T* W = reinterpret_cast<const T*>(a.phi.W) + (size_t)hset * M * DH;
  const float* bias = a.phi.b + (size_t)hset * M;

  // chunks [c_first, c_begin) only build the state; chunks [c_begin, c_end) are scanned
  int c_first, c_begin, c_end, t_end;
  if (state_run) {
    c_first = part * a.piece_chunks;
    c_end = min(a.split / 64, c_first + a.piece_chunks);
    c_begin = c_end;
    t_end = 0;
  } else if (a.staged) {
    c_first = part == 0 ? a.pc_first[0] : a.pc_first[1];
    c_begin = part == 0 ? a.pc_begin[0] : a.pc_begin[1];
    c_end = part == 0 ? a.pc_end[0] : a.pc_end[1];
    t_end = min(n, 64 * c_end);
  } else {
    const int t_begin = part == 0 ? 0 : a.split;
    t_end = part == a.parts - 1 ? n : a.split;
    c_begin = t_begin / 64;
    c_end = (t_end + 63) / 64;
    c_first = (part > 0 && a.state_in != nullptr) ? c_begin : 0;
  }
  // part 1 of the scan launch starts from the state of the first c_first chunks: the
  // sum of the pieces, in piece order (a staged part from the sum of its first npc)
  const int npc = a.staged ? (part == 0 ? a.pseed[0] : a.pseed[1]) : a.pieces;
  const bool seeded = !state_run && (a.staged ? npc > 0 : c_first > 0);
  const float* seed = seeded ? a.state_in + (size_t)head * a.pieces * C::STATE : nullptr;

  // Q, K, V rows of chunk cc and the output rows of chunk cc as range-checked
  // buffers: rows at or past n (t_end for the output) read as 0 and are not written.
  auto rows_of = [&](const void* base, int cc, int t_lim) {
    const char* p = reinterpret_cast<const char*>(base) + (hoff + (size_t)64 * cc * DH) * SZ;
    // uniform, and kept in a scalar register: a vector-held record count would make
    // every buffer access a readfirstlane loop
    const int rows = __builtin_amdgcn_readfirstlane(max(0, min(64, t_lim - 64 * cc)));
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(p), (short)0, rows * DH * SZ, kBufferFlags);
  };

  // W fragments into LDS; P (above-diagonal blocks stay zero) and z cleared
  for (int i = tid; i < (PF ? 0 : MB * KS * kWave); i += C::NT) {
    const int l = i % kWave, ks = (i / kWave) % KS, mb = i / (kWave * KS);
    const int p = 16 * mb + l % 16;
    Frag<T> f;
    if (p < M) load8(f, W + (size_t)p * DH + 32 * ks + 8 * (l / 16));
    else f.zero();
    store8(&sm.wfr[mb][ks][l][0], f);
  }
  for (int i = tid; i < 64 * SP / 4; i += C::NT) reinterpret_cast<int*>(sm.pm)[i] = 0;
  // z_{c_first - 1} in the slot that chunk c_first's denominators read; the other 0
  for (int i = tid; i < 2 * FP; i += C::NT) {
    float zv = 0.0f;
    if (seeded && i / FP == ((c_first + 1) & 1))
      for (int pc = 0; pc < npc; ++pc) zv += seed[(size_t)pc * C::STATE + C::SF + i % FP];
    (&sm.zs[0][0])[i] = (T)zv;
  }
  if constexpr (!PF)
    for (int i = tid; i < 16 * MB; i += C::NT) sm.bias[i] = i < M ? bias[i] : 0.0f;

  if (wave >= NMS) {
    if constexpr (PF) {
      // ============================================== map waves, features given
      // Map wave b moves rows 16 b .. 16 b + 15 of the next chunk: phi(Q) copied
      // token-major (feature f at position f), phi(K) transposed in registers (feature f
      // to phi(K)^T row krow(f)), a share of V, and running sums of its key rows'
      // features for z.  Lane (tg, fc) holds features 8 fc .. 8 fc + 7 of TPL consecutive
      // tokens.
      __builtin_amdgcn_s_setprio(3);
      constexpr int CPR = FP / 8, TG = kWave / CPR, TPL = 16 / TG;
      const int rb = wave - NMS, mtid = tid - 64 * NMS;
      const int fc = lane % CPR, tg = lane / CPR;
      const int t0 = 16 * rb + TPL * tg;  // this lane's first token in the chunk
      i32x4 qv[TPL], kv[TPL];
      i32x4 vr[C::VPT];
      float zrun[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) zrun[e] = 0.0f;
      if (seeded && rb == 0 && tg == 0)  // the prefix's z enters through map wave 0
        for (int pc = 0; pc < npc; ++pc)
#pragma unroll
          for (int e = 0; e < 8; ++e) zrun[e] += seed[(size_t)pc * C::STATE + C::SF + 8 * fc + e];
      auto load_feat = [&](i32x4 (&dst)[TPL], const void* X, int cc, bool live) {
        const char* base = reinterpret_cast<const char*>(X) + ((size_t)head * n + (size_t)64 * cc) * FP * SZ;
        const int rows = __builtin_amdgcn_readfirstlane(max(0, min(64, (live ? n : 0) - 64 * cc)));
        const auto rs =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), (short)0, rows * FP * SZ, kBufferFlags);
#pragma unroll
        for (int k = 0; k < TPL; ++k)
          dst[k] = __builtin_bit_cast(
              i32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, ((t0 + k) * FP + 8 * fc) * SZ, 0, 0));
      };
      auto load_v = [&](int cc) {
        const auto rs = rows_of(a.V, cc, n);
#pragma unroll
        for (int q = 0; q < C::VPT; ++q)
          vr[q] = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, 16 * (mtid + 256 * q), 0, 0));
      };
      auto store_v = [&]() {
#pragma unroll
        for (int q = 0; q < C::VPT; ++q) {
          const int cidx = mtid + 256 * q;
          const int tt = cidx / CPV, cg = cidx % CPV;
          *reinterpret_cast<i32x4*>(&sm.vt[tt * DH + swz_v<CPV>(tt, cg) * VE]) = vr[q];
        }
      };
      auto write_q = [&]() {
#pragma unroll
        for (int k = 0; k < TPL; ++k) *reinterpret_cast<i32x4*>(sm.phq + (t0 + k) * SQ + 16 * fc) = qv[k];
      };
      // feature 8 fc + e of the TPL tokens: one store into its phi(K)^T row
      auto write_k = [&]() {
        typedef __attribute__((ext_vector_type(TPL))) __bf16 bf16xT;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          bf16xT col;
#pragma unroll
          for (int k = 0; k < TPL; ++k) col[k] = __builtin_bit_cast(bf16x8, kv[k])[e];
          *reinterpret_cast<bf16xT*>(sm.phk + krow(8 * fc + e) * SK + t0 * SZ) = col;
        }
      };
      auto add_z = [&]() {
#pragma unroll
        for (int k = 0; k < TPL; ++k)
#pragma unroll
          for (int e = 0; e < 8; ++e) zrun[e] += (float)__builtin_bit_cast(bf16x8, kv[k])[e];
      };
      // z over this wave's key rows through the chunk just written (lanes of one fc summed)
      auto write_z = [&]() {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          float zz = sum_xor32(zrun[e]);
          if constexpr (TG == 4) zz = sum_xor16(zz);
          if (tg == 0) sm.zp[rb][8 * fc + e] = zz;
        }
      };
      auto sum_z = [&](int slot) {
        constexpr int FW = FP / 4;
#pragma unroll
        for (int f0 = 0; f0 < FW; f0 += kWave) {
          const int f = FW * rb + f0 + lane;
          if (f0 + lane < FW) sm.zs[slot][f] = (T)(((sm.zp[0][f] + sm.zp[1][f]) + sm.zp[2][f]) + sm.zp[3][f]);
        }
      };
      if constexpr (ST) {
        // state launch: phi(K) and V only (z is summed by matrix wave 0)
        load_feat(kv, a.phik, c_first, c_first < c_end);
        load_v(c_first);
        __syncthreads();  // cleared P and z
        write_k();
        store_v();
        load_feat(kv, a.phik, c_first + 1, c_first + 1 < c_end);
        load_v(c_first + 1);
        for (int c = c_first; c < c_end; ++c) {
          const int cn = c + 1;
          __syncthreads();  // B1
          __syncthreads();  // B2
          if (cn < c_end) {
            write_k();
            store_v();
          }
          load_feat(kv, a.phik, cn + 1, cn + 1 < c_end);
          load_v(cn + 1);
        }
      } else {
        const bool q0 = c_first >= c_begin;
        load_feat(qv, a.phiq, c_first, q0 && c_first < c_end);
        load_feat(kv, a.phik, c_first, c_first < c_end);
        load_v(c_first);
        __syncthreads();  // cleared P and z
        if (q0) write_q();
        write_k();
        add_z();
        write_z();  // z through chunk c_first
        store_v();
        load_feat(qv, a.phiq, c_first + 1, c_first + 1 >= c_begin && c_first + 1 < c_end);
        load_feat(kv, a.phik, c_first + 1, c_first + 1 < c_end);
        load_v(c_first + 1);
        // iteration c: chunk c + 1's rows (loaded one iteration ahead) are written after B2
        for (int c = c_first; c < c_end; ++c) {
          const int cn = c + 1;
          __syncthreads();  // B1: chunk c's tiles are in LDS; zp holds z through chunk c
          sum_z(c & 1);
          __syncthreads();  // B2: chunk c's phi tiles and V are no longer read
          const bool kn = cn < c_end, qn = kn && cn >= c_begin;
          if (kn) {
            if (qn) write_q();
            write_k();
            add_z();
            write_z();  // z through chunk c + 1
            store_v();
          }
          load_feat(qv, a.phiq, cn + 1, kn && cn + 1 >= c_begin && cn + 1 < c_end);
          load_feat(kv, a.phik, cn + 1, cn + 1 < c_end);
          load_v(cn + 1);
        }
      }
    } else {
      // ============================================================== map waves
      // The map work is a chain of dependent table lookups: its LDS requests are issued
      // ahead of the matrix waves' bursts of operand reads.
      __builtin_amdgcn_s_setprio(3);
      const int rb = wave - NMS;  // rows 16 rb .. 16 rb + 15 of every chunk, all projections
      const int mtid = tid - 64 * NMS;
      const bool pad_proj = 16 * MB > M;  // padded projections exist (phi(K) of them is set to 0)
      // byte offsets of this lane's pieces
      const int x_off = ((16 * rb + r) * DH + 8 * g) * SZ;  // its slice of a Q or K row in a chunk
      // phi(Q) of token 16 rb + r, projection 16 mb + 4 g + j, channel l: feature
      // feat(4 g, 0) + feat(16 mb, l) + j
      char* q_dst = sm.phq + (16 * rb + r) * SQ + feat<MB>(4 * g, 0) * SZ;
      // phi(K)^T row 16 (mb + MB l) + r (projection 16 mb + r, channel l), tokens 16 rb + 4 g ..
      char* k_dst = sm.phk + r * SK + (16 * rb + 4 * g) * SZ;
      Frag<T> xq[KS], xk[KS];  // query and key rows of the next chunk to map
      i32x4 vr[C::VPT];        // this thread's share of V of the next chunk
      auto load_rows = [&](Frag<T> (&xf)[KS], const void* X, int cc, bool live) {
        const auto rs = rows_of(X, cc, live ? n : 0);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) buf_load8(xf[ks], rs, x_off + 32 * ks * SZ);
      };
      auto load_v = [&](int cc) {
        const auto rs = rows_of(a.V, cc, n);
#pragma unroll
        for (int q = 0; q < C::VPT; ++q)
          vr[q] = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, 16 * (mtid + 256 * q), 0, 0));
      };
      auto store_v = [&]() {
#pragma unroll
        for (int q = 0; q < C::VPT; ++q) {
          const int cidx = mtid + 256 * q;
          const int tt = cidx / CPV, cg = cidx % CPV;
          *reinterpret_cast<i32x4*>(&sm.vt[tt * DH + swz_v<CPV>(tt, cg) * VE]) = vr[q];
        }
      };
      // W fragments and biases of all projections, held in registers
      Frag<T> wreg[MB][KS];
      f32x4 bq[MB], bk[MB];
      // u for the 16 rows: query rows as u^T = W X^T (lane: projections 16 mb + 4 g + j
      // of token r), key rows as u = X W^T (lane: projection 16 mb + r of tokens 4 g + j);
      // the accumulators start at the biases
      auto project = [&](const Frag<T> (&xf)[KS], bool isq, float (&uu)[4 * MB]) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          f32x4 acc = isq ? bq[mb] : bk[mb];
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            if (isq) mma(acc, wreg[mb][ks], xf[ks]);
            else mma(acc, xf[ks], wreg[mb][ks]);
          }
#pragma unroll
          for (int j = 0; j < 4; ++j) uu[4 * mb + j] = acc[j];
        }
      };
      // phi of this lane's 4 MB values u, as Pack4<T> per (block, channel) (the four j
      // in order), from the values and their segment offsets; query and key rows
      Pack4<T> phq_r[MB][L], phk_r[MB][L];
      auto eval_all = [&](Pack4<T> (&ph)[MB][L], const float (&uu)[4 * MB], const unsigned (&off)[4 * MB],
                          float floor) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int jp = 0; jp < 2; ++jp) {
            const int i0 = 4 * mb + 2 * jp;
            float y0[L], y1[L];
            pwl_eval_off(sm.tab, off[i0], floor, uu[i0], y0);
            pwl_eval_off(sm.tab, off[i0 + 1], floor, uu[i0 + 1], y1);
#pragma unroll
            for (int l = 0; l < L; ++l) ph[mb][l].set2(2 * jp, y0[l], y1[l]);
          }
      };
      auto write_q = [&]() {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int l = 0; l < L; ++l) phq_r[mb][l].store(q_dst + feat<MB>(16 * mb, l) * SZ);
      };
      auto write_k = [&]() {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int l = 0; l < L; ++l) phk_r[mb][l].store(k_dst + 16 * (mb + MB * l) * SK);
      };
      // z over this wave's key rows: tile mb rows = projections 16 mb + 4 g + jj,
      // column l = channel l, accumulated from phi(K) fragments (channels 2q, 2q + 1 of
      // tokens 4 g .. 4 g + 3) times one-hot columns
      f32x4 zacc[MB];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) zacc[mb] = zero4();
      if (seeded && rb == 0 && r < L) {  // the prefix's z enters through map wave 0
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
            for (int pc = 0; pc < npc; ++pc)
              zacc[mb][jj] += seed[(size_t)pc * C::STATE + C::SF + feat<MB>(16 * mb + 4 * g, r) + jj];
      }
      auto add_z = [&]() {
#pragma unroll
        for (int q = 0; q < L / 2; ++q) {
          Frag<T> oh;
          const float lo = r == 2 * q ? 1.0f : 0.0f, hi = r == 2 * q + 1 ? 1.0f : 0.0f;
          oh.set2(0, lo, lo);
          oh.set2(2, lo, lo);
          oh.set2(4, hi, hi);
          oh.set2(6, hi, hi);
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) {
            Frag<T> kf;
            phk_r[mb][2 * q].to_frag(kf, 0);
            phk_r[mb][2 * q + 1].to_frag(kf, 4);
            mma(zacc[mb], kf, oh);
          }
        }
      };
      auto write_z = [&]() {
        if (r < L) {
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) {
            float* zp = &sm.zp[rb][feat<MB>(16 * mb + 4 * g, r)];
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) zp[jj] = zacc[mb][jj];
          }
        }
      };
      // the four row-block parts summed in a fixed order, this wave's quarter of the features
      auto sum_z = [&](int slot) {
        constexpr int FW = FP / 4;
#pragma unroll
        for (int f0 = 0; f0 < FW; f0 += kWave) {
          const int f = FW * rb + f0 + lane;
          if (f0 + lane < FW) sm.zs[slot][f] = (T)(((sm.zp[0][f] + sm.zp[1][f]) + sm.zp[2][f]) + sm.zp[3][f]);
        }
      };
      // query rows are needed from chunk c_begin on, key rows and V from chunk c_first
      load_rows(xq, a.Q, c_first, c_first >= c_begin && c_first < c_end);
      load_rows(xk, a.K, c_first, c_first < c_end);
      load_v(c_first);
      __syncthreads();  // tables, W fragments, cleared P and z
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) load8(wreg[mb][ks], &sm.wfr[mb][ks][lane][0]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          bq[mb][j] = sm.bias[16 * mb + 4 * g + j];
          bk[mb][j] = sm.bias[16 * mb + r];
        }
      }
      const int steps = __builtin_amdgcn_readfirstlane(sm.tab.steps);
      const int nodes = __builtin_amdgcn_readfirstlane(pwl_nodes(sm.tab));
      const unsigned zoff = 4u * sm.tab.zero_seg;
      const float tfloor = sm.tab.floor;
      // u of the query rows and the key rows of one chunk and their segment offsets
      float uq[4 * MB], uk[4 * MB];
      unsigned oq[4 * MB], ok[4 * MB];
      // projections of the rows held in xq, xk and the searches, as one batch when the
      // query rows are live, so that their lookups overlap
      auto project_search = [&](auto qlive) {
        constexpr bool kQ = decltype(qlive)::value;
        if constexpr (kQ) {
          project(xq, true, uq);
          project(xk, false, uk);
          float uu[8 * MB];
          unsigned oo[8 * MB];
#pragma unroll
          for (int i = 0; i < 4 * MB; ++i) {
            uu[i] = uq[i];
            uu[4 * MB + i] = uk[i];
          }
          pwl_search_any(sm.tab, steps, nodes, uu, oo);
#pragma unroll
          for (int i = 0; i < 4 * MB; ++i) {
            oq[i] = oo[i];
            ok[i] = oo[4 * MB + i];
          }
        } else {
          project(xk, false, uk);
          pwl_search_any(sm.tab, steps, nodes, uk, ok);
        }
        if (pad_proj) {  // padded projections of the key rows select the all-zero segment
#pragma unroll
          for (int i = 0; i < 4 * MB; ++i)
            if (16 * (i / 4) + r >= M) ok[i] = zoff;
        }
      };
      // phi of the rows held in xq, xk (the query rows when live) into phq_r, phk_r, and
      // the key rows added to z
      auto map_rows = [&](auto qlive, int cc) {
        project_search(qlive);
        if constexpr (ST) {  // key rows at or past n (a state of the whole sequence) add nothing
#pragma unroll
          for (int i = 0; i < 4 * MB; ++i)
            if (64 * cc + 16 * rb + 4 * g + i % 4 >= n) ok[i] = zoff;
        }
        if constexpr (decltype(qlive)::value) eval_all(phq_r, uq, oq, tfloor);
        eval_all(phk_r, uk, ok, tfloor);
        if constexpr (!ST) add_z();  // (the state launch's z comes from matrix wave 0)
      };
      if constexpr (ST) {
        // State launch: every chunk is state-only; z is summed by matrix wave 0 along
        // with its slice of S (one-hot products here would lengthen the map waves'
        // chain, which sets this launch's pace).  (Mapping the key rows of two chunks as
        // one batch made this launch slower: 186 against 159 us.)
        map_rows(std::false_type{}, c_first);
        load_rows(xq, a.Q, c_first + 1, false);
        load_rows(xk, a.K, c_first + 1, c_first + 1 < c_end);
        write_k();
        store_v();
        load_v(c_first + 1);
        for (int c = c_first; c < c_end; ++c) {
          const int cn = c + 1;
          __syncthreads();  // B1
          const bool kn = cn < c_end;
          if (kn) map_rows(std::false_type{}, cn);
          load_rows(xq, a.Q, cn + 1, false);  // issued on every path (see the scan launch)
          load_rows(xk, a.K, cn + 1, kn);
          __syncthreads();  // B2
          if (kn) {
            write_k();
            store_v();
          }
          load_v(cn + 1);
        }
      } else {
        // chunk c_first
        if (c_first >= c_begin) map_rows(std::true_type{}, c_first);
        else map_rows(std::false_type{}, c_first);
        load_rows(xq, a.Q, c_first + 1, c_first + 1 >= c_begin && c_first + 1 < c_end);
        load_rows(xk, a.K, c_first + 1, c_first + 1 < c_end);
        if (c_first >= c_begin) write_q();
        write_k();
        write_z();  // z through chunk c_first
        store_v();
        load_v(c_first + 1);

        // Iteration c: between B1 and B2 the matrix waves read chunk c's tiles while this
        // wave maps chunk c + 1 (rows fetched one chunk ahead) into registers; after B2 it
        // writes chunk c + 1's tiles, V and z.
        for (int c = c_first; c < c_end; ++c) {
          const int cn = c + 1;
          __syncthreads();  // B1: chunk c's tiles are in LDS; zp holds z through chunk c
          sum_z(c & 1);
          const bool kn = cn < c_end, qn = kn && cn >= c_begin;
          // phi(Q) before B2; the key rows are only projected and searched here and
          // evaluated after B2, where the matrix waves' work is shorter
          if (qn) {
            project_search(std::true_type{});
            eval_all(phq_r, uq, oq, tfloor);
          } else if (kn) {
            project_search(std::false_type{});
          }
          // the loads are issued on every path (past the end as empty buffers, which read
          // nothing), so that the waits for them count the same loads on every path
          load_rows(xq, a.Q, cn + 1, kn && cn + 1 >= c_begin);
          load_rows(xk, a.K, cn + 1, kn);
          __syncthreads();  // B2: chunk c's phi tiles and V are no longer read
          if (kn) {
            if (qn) write_q();
            eval_all(phk_r, uk, ok, tfloor);
            add_z();
            write_k();
            write_z();  // z through chunk c + 1
            store_v();
          }
          load_v(cn + 1);
        }
      }
    }
  } else {
    // =========================================================== matrix waves
    const int mw = wave;
    const bool active = mw < NMW;
    // byte offsets of this lane's operands (every access adds a constant)
    const char* q_src = sm.phq + r * SQ + 8 * g * SZ;  // phi(Q) row r, features 8 g ..
    const char* k_src = sm.phk + r * SK + 8 * g * SZ;  // phi(K)^T row r, tokens 8 g ..
    const char* p_src = sm.pm + r * SP + 8 * g * SZ;   // P row r, keys 8 g ..
    char* p_dst = sm.pm + r * SP + 4 * g * SZ;         // P row r, keys 4 g ..
    const int i16 = lane % 16;
    // transposed reads of phi(K)^T rows 4 g + kk (kk = 0..3), token column i16 (see
    // load_tr4_rows for the two address forms)
    const char* kt_src = sizeof(T) == 2 ? sm.phk + (4 * g + i16 / 4) * SK + 4 * (i16 % 4) * SZ
                                        : sm.phk + 4 * g * SK + i16 * SZ;
    const T* zs0 = &sm.zs[0][8 * g];
    f32x4 sacc[CBW][RB];
    // state launch: z of the chunks, summed by matrix wave 0 from its phi(K)^T fragments
    f32x4 zst[ST ? RB : 1];
#pragma unroll
    for (int i = 0; i < (ST ? RB : 1); ++i) zst[i] = zero4();
    Frag<T> ones;
    ones.fill(1.0f);
    // the state piece layout: S tile (x, b) of matrix wave mw at (mw CBW + x) RB + b,
    // lane-major 16-byte entries
    const size_t s_off = ((size_t)mw * CBW * RB * kWave + lane) * 4;
#pragma unroll
    for (int x = 0; x < CBW; ++x)
#pragma unroll
      for (int i = 0; i < RB; ++i) {
        sacc[x][i] = zero4();
        if (seeded && active)
          for (int pc = 0; pc < npc; ++pc)
            sacc[x][i] += *reinterpret_cast<const f32x4*>(seed + (size_t)pc * C::STATE + s_off +
                                                          (size_t)(x * RB + i) * kWave * 4);
      }
    f32x4 num[CBW][4];  // num^T of the chunk being scanned
#pragma unroll
    for (int x = 0; x < CBW; ++x)
#pragma unroll
      for (int i = 0; i < 4; ++i) num[x][i] = zero4();
    __syncthreads();  // tables, W fragments, cleared P and z
    // (the bf16 tables' coefficient rows carry a power-of-two scale, which eps takes too)
    float eps = a.eps;
    if constexpr (!PF) eps = ldexpf(a.eps, 2 * sm.tab.scale_exp);

    // P^T blocks (query block i >= key block j): rows = key tokens 16 j + 4 g + jj,
    // column = query token 16 i + r, for CNT query blocks i0 .. i0 + CNT - 1 that share
    // key block j, so that phi(K_j) is read once per run.  k-slot (g, e) of fragment kf
    // is feature 32 kf + 8 g + e: phi(Q) positions 32 kf + 8 g + e, phi(K)^T rows
    // 32 kf + 16 (e / 4) + 4 g + e % 4.  Operands of kf + 1 are read while kf multiplies.
    // P^T block (j, i) to LDS (entries above the diagonal zeroed) and its row sums
    auto p_store = [&](f32x4 p, int j, int i) {
      if (i == j) {
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
          if (4 * g + jj > r) p[jj] = 0.0f;
      }
      store4(reinterpret_cast<T*>(p_dst + 16 * i * SP + 16 * j * SZ), p[0], p[1], p[2], p[3]);
      float rs = (p[0] + p[1]) + (p[2] + p[3]);
      rs = sum_xor32(sum_xor16(rs));
      if (g == 0) sm.denp[j][16 * i + r] = rs;
    };
    auto p_run = [&](auto cnt, int j, int i0) {
      constexpr int CNT = decltype(cnt)::value;
      f32x4 pacc[CNT];
#pragma unroll
      for (int b = 0; b < CNT; ++b) pacc[b] = zero4();
      Frag<T> kfr[2], qb[2][CNT];
      auto rd = [&](int kf, int s) {
        load_tr4_rows(kfr[s], 0, kt_src + 32 * kf * SK + 16 * j * SZ, SK);
        load_tr4_rows(kfr[s], 4, kt_src + (32 * kf + 16) * SK + 16 * j * SZ, SK);
#pragma unroll
        for (int b = 0; b < CNT; ++b) lds8(qb[s][b], q_src + 16 * (i0 + b) * SQ + 32 * kf * SZ);
      };
      rd(0, 0);
#pragma unroll
      for (int kf = 0; kf < NF; ++kf) {
        if (kf + 1 < NF) rd(kf + 1, (kf + 1) & 1);
#pragma unroll
        for (int b = 0; b < CNT; ++b) mma(pacc[b], kfr[kf & 1], qb[kf & 1][b]);
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int b = 0; b < CNT; ++b) p_store(pacc[b], j, i0 + b);
    };
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using I3 = std::integral_constant<int, 3>;
    using I4 = std::integral_constant<int, 4>;
    // phi(Q_c) z_{c-1} for query block i (every row of the z operand is z, so every
    // accumulator row is the answer)
    auto den_run = [&](const T* zprev, int i) {
      f32x4 dacc = zero4();
#pragma unroll
      for (int kf = 0; kf < NF; ++kf) {
        Frag<T> za, qb;
        lds8(za, reinterpret_cast<const char*>(zprev + 32 * kf));
        lds8(qb, q_src + 16 * i * SQ + 32 * kf * SZ);
        mma(dacc, za, qb);
        if (kf % 2 == 1) __builtin_amdgcn_sched_barrier(0);
      }
      if (g == 0) sm.deni[16 * i + r] = dacc[0];
    };

    // num^T = S_{c-1}^T phi(Q_c)^T: accumulator tiles 2 kf, 2 kf + 1 of S are the
    // k-fragment kf of S^T (slot (g, e) = feature 32 kf + 8 g + e); phi(Q) fragments
    // (step kf, block i) are read in that order kPre ahead of their use
    auto readout = [&]() {
#pragma unroll
      for (int x = 0; x < CBW; ++x)
#pragma unroll
        for (int i = 0; i < 4; ++i) num[x][i] = zero4();
      constexpr int kPre = 4;
      auto q_read = [&](Frag<T>& f, int idx) { lds8(f, q_src + 16 * (idx % 4) * SQ + 32 * (idx / 4) * SZ); };
      Frag<T> qb[kPre];
#pragma unroll
      for (int p = 0; p < kPre; ++p) q_read(qb[p], p);
#pragma unroll
      for (int kf = 0; kf < NF; ++kf) {
        Frag<T> sa[CBW];
#pragma unroll
        for (int x = 0; x < CBW; ++x) {
          sa[x].set2(0, sacc[x][2 * kf][0], sacc[x][2 * kf][1]);
          sa[x].set2(2, sacc[x][2 * kf][2], sacc[x][2 * kf][3]);
          sa[x].set2(4, sacc[x][2 * kf + 1][0], sacc[x][2 * kf + 1][1]);
          sa[x].set2(6, sacc[x][2 * kf + 1][2], sacc[x][2 * kf + 1][3]);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int idx = 4 * kf + i;
          const Frag<T> qa = qb[idx % kPre];
          if (idx + kPre < 4 * NF) q_read(qb[idx % kPre], idx + kPre);
#pragma unroll
          for (int x = 0; x < CBW; ++x) mma(num[x][i], sa[x], qa);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    };

    // The readout, this wave's P^T runs (key block J0, query blocks I0 .. I0 + C0 - 1,
    // and J1, I1 .. I1 + C1 - 1) and its den block ID in one pass over phi(Q_c): every
    // phi(Q) fragment is read once and is the B operand of all three.  phi(K)^T and z
    // fragments of step kf are read at its start and first used after its readout
    // products (one buffer: registers are at the limit).
    auto front = [&](const T* zprev, auto j0c, auto i0c, auto c0c, auto j1c, auto i1c, auto c1c, auto idc) {
      constexpr int J0 = decltype(j0c)::value, I0 = decltype(i0c)::value, C0 = decltype(c0c)::value;
      constexpr int J1 = decltype(j1c)::value, I1 = decltype(i1c)::value, C1 = decltype(c1c)::value;
      constexpr int ID = decltype(idc)::value;
      f32x4 pa0[C0], pa1[C1 > 0 ? C1 : 1], dacc = zero4();
#pragma unroll
      for (int b = 0; b < C0; ++b) pa0[b] = zero4();
#pragma unroll
      for (int b = 0; b < C1; ++b) pa1[b] = zero4();
#pragma unroll
      for (int x = 0; x < CBW; ++x)
#pragma unroll
        for (int i = 0; i < 4; ++i) num[x][i] = zero4();
      constexpr int kPre = 4;
      auto q_read = [&](Frag<T>& f, int idx) { lds8(f, q_src + 16 * (idx % 4) * SQ + 32 * (idx / 4) * SZ); };
      Frag<T> qb[kPre], k0, k1, za;
#pragma unroll
      for (int p = 0; p < kPre; ++p) q_read(qb[p], p);
#pragma unroll
      for (int kf = 0; kf < NF; ++kf) {
        load_tr4_rows(k0, 0, kt_src + 32 * kf * SK + 16 * J0 * SZ, SK);
        load_tr4_rows(k0, 4, kt_src + (32 * kf + 16) * SK + 16 * J0 * SZ, SK);
        if constexpr (C1 > 0) {
          load_tr4_rows(k1, 0, kt_src + 32 * kf * SK + 16 * J1 * SZ, SK);
          load_tr4_rows(k1, 4, kt_src + (32 * kf + 16) * SK + 16 * J1 * SZ, SK);
        }
        lds8(za, reinterpret_cast<const char*>(zprev + 32 * kf));
        Frag<T> sa[CBW];
#pragma unroll
        for (int x = 0; x < CBW; ++x) {
          sa[x].set2(0, sacc[x][2 * kf][0], sacc[x][2 * kf][1]);
          sa[x].set2(2, sacc[x][2 * kf][2], sacc[x][2 * kf][3]);
          sa[x].set2(4, sacc[x][2 * kf + 1][0], sacc[x][2 * kf + 1][1]);
          sa[x].set2(6, sacc[x][2 * kf + 1][2], sacc[x][2 * kf + 1][3]);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int idx = 4 * kf + i;
          const Frag<T> qa = qb[idx % kPre];
          if (idx + kPre < 4 * NF) q_read(qb[idx % kPre], idx + kPre);
#pragma unroll
          for (int x = 0; x < CBW; ++x) mma(num[x][i], sa[x], qa);
          if (i >= I0 && i < I0 + C0) mma(pa0[i - I0], k0, qa);
          if constexpr (C1 > 0)
            if (i >= I1 && i < I1 + C1) mma(pa1[i - I1], k1, qa);
          if (i == ID) mma(dacc, za, qa);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int b = 0; b < C0; ++b) p_store(pa0[b], J0, I0 + b);
#pragma unroll
      for (int b = 0; b < C1; ++b) p_store(pa1[b], J1, I1 + b);
      if (g == 0) sm.deni[16 * ID + r] = dacc[0];
    };
    using I0c = std::integral_constant<int, 0>;

    // Iteration c: between B1 and B2 the readout of chunk c from S_{c-1}, the P^T and
    // denominator blocks, the V fragments and the S update; after B2, V^T P^T and the
    // output rows.
    for (int c = c_first; c < c_end; ++c) {
      const bool scan = c >= c_begin;
      __syncthreads();  // B1: phi(Q_c), phi(K_c), V_c and z_{c-1} are in LDS
      Frag<T> vf[CBW][2];  // V columns 16 (CBW mw + x) + r, tokens 32 ks + 8 g + e
      if (active) {
        if (!ST && scan) {
          const T* zprev = zs0 + ((c + 1) & 1) * FP;  // z_{c-1}
          // the ten P^T blocks and four den blocks spread over the matrix waves
          if constexpr (NMW == 4) {
            if (mw == 0) front(zprev, I0c{}, I0c{}, I3{}, I0c{}, I0c{}, I0c{}, I2{});
            else if (mw == 1) front(zprev, I0c{}, I3{}, I1{}, I3{}, I3{}, I1{}, I3{});
            else if (mw == 2) front(zprev, I1{}, I1{}, I3{}, I0c{}, I0c{}, I0c{}, I0c{});
            else front(zprev, I2{}, I2{}, I2{}, I0c{}, I0c{}, I0c{}, I1{});
          } else {
            readout();
            if (mw == 0) { p_run(I4{}, 0, 0); p_run(I2{}, 2, 2); }
            else { p_run(I3{}, 1, 1); p_run(I1{}, 3, 3); }
            den_run(zprev, mw);
            den_run(zprev, mw + 2);
          }
        }
#pragma unroll
        for (int x = 0; x < CBW; ++x)
#pragma unroll
          for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int h = 0; h < 2; ++h)
              load_tr4_at(vf[x][ks], 4 * h, lane, [&](int kk, int col) {
                const int t = 32 * ks + 8 * g + 4 * h + kk, cc = 16 * (CBW * mw + x) + col;
                return &sm.vt[t * DH + swz_v<CPV>(t, cc / VE) * VE + cc % VE];
              });
        // S += phi(K_c)^T V_c, S row block b = phi(K)^T rows 16 b .. 16 b + 15;
        // fragments read kPre ahead
        constexpr int kPre = 4;
        auto ka_read = [&](Frag<T>& f, int idx) { lds8(f, k_src + 16 * (idx / 2) * SK + 32 * (idx % 2) * SZ); };
        Frag<T> kb[kPre];
#pragma unroll
        for (int p = 0; p < kPre; ++p) ka_read(kb[p], p);
#pragma unroll
        for (int idx = 0; idx < 2 * RB; ++idx) {
          const Frag<T> ka = kb[idx % kPre];
          if (idx + kPre < 2 * RB) ka_read(kb[idx % kPre], idx + kPre);
#pragma unroll
          for (int x = 0; x < CBW; ++x) mma(sacc[x][idx / 2], ka, vf[x][idx % 2]);
          if constexpr (ST)
            if (mw == 0) mma(zst[idx / 2], ka, ones);  // z: every column of the tile is z
        }
      }
      __syncthreads();  // B2: P and the den parts are in LDS
      if (!ST && active && scan) {
        // num^T += V^T P^T over the key tokens at or before each query block
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int ks = 0; ks < 2; ++ks)
            if (2 * ks <= i) {
              Frag<T> pb;
              lds8(pb, p_src + 16 * i * SP + 32 * ks * SZ);
#pragma unroll
              for (int x = 0; x < CBW; ++x) mma(num[x][i], vf[x][ks], pb);
            }
        const auto ro = rows_of(a.out, c, t_end);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int q = 16 * i + r;
          float den = sm.deni[q];
#pragma unroll
          for (int j = 0; j <= i; ++j) den += sm.denp[j][q];
          const float rinv = __builtin_amdgcn_rcpf(den + eps);
#pragma unroll
          for (int x = 0; x < CBW; ++x)
            buf_store4<T>(ro, (q * DH + 16 * (CBW * mw + x) + 4 * g) * SZ, num[x][i][0] * rinv,
                          num[x][i][1] * rinv, num[x][i][2] * rinv, num[x][i][3] * rinv);
        }
      }
    }
    if (ST && active) {
      float* so = a.state_out + (size_t)(head * a.pieces + part) * C::STATE + s_off;
#pragma unroll
      for (int x = 0; x < CBW; ++x)
#pragma unroll
        for (int i = 0; i < RB; ++i) *reinterpret_cast<f32x4*>(so + (size_t)(x * RB + i) * kWave * 4) = sacc[x][i];
      if constexpr (ST) {
        if (mw == 0 && r == 0) {  // z of the piece, by internal feature
          float* zo = a.state_out + (size_t)(head * a.pieces + part) * C::STATE + C::SF;
#pragma unroll
          for (int b = 0; b < RB; ++b)
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) zo[krow_inv(16 * b + 4 * g + jj)] = zst[b][jj];
        }
      }
    }
    if constexpr (!ST && !PF) {
      // staged: the final state of this part as piece `part` of its head.  z is the sum
      // of the map waves' row-block partials (fp32, through the last chunk; the last
      // were written before the last chunk's first barrier), in a fixed order.
      if (a.state_fin != nullptr && active) {
        float* so = a.state_fin + (size_t)(head * a.pieces + part) * C::STATE;
#pragma unroll
        for (int x = 0; x < CBW; ++x)
#pragma unroll
          for (int i = 0; i < RB; ++i)
            *reinterpret_cast<f32x4*>(so + s_off + (size_t)(x * RB + i) * kWave * 4) = sacc[x][i];
        for (int f = kWave * mw + lane; f < FP; f += kWave * NMW)
          so[C::SF + f] = ((sm.zp[0][f] + sm.zp[1][f]) + sm.zp[2][f]) + sm.zp[3][f];
      }
    }
  }
}

// State export: the state launch's pieces summed in piece order and written as
// S [M*L][d], z [M*L] (fp32, feature i*L + l, the coefficient rows' power-of-two scale
// removed), or added to them.  A piece holds the matrix waves' S tiles, lane-major
// (tile (mw CBW + x) RB + b: rows krow(f) = 16 b + 4 g + jj, column 16 (CBW mw + x) + r
// of lane 16 g + r), then z by internal feature.
template <typename T, int DH, int L, int MB>
__global__ __launch_bounds__(256) void causal_state_export_kernel(CausalArgs a) {
  using C = CsCfg<T, DH, L, MB>;
  const int head = blockIdx.x;  // blockIdx.y: a slice of the head's elements
  const int hset = a.phi.per_head ? head % a.H : 0;
  const PwlHeader hd = *reinterpret_cast<const PwlHeader*>(a.phi.tables + (size_t)hset * kTableBytes + kTabHeader);
  const float unscale = sizeof(T) == 2 ? ldexpf(1.0f, -hd.scale_exp) : 1.0f;
  const int M = a.phi.M;
  const float* pc = a.state_out + (size_t)head * a.pieces * C::STATE;
  float* S = a.export_S + (size_t)head * M * L * DH;
  float* z = a.export_z + (size_t)head * M * L;
  // internal feature f -> projection and channel (the inverse of feat<MB>)
  auto proj_chan = [](int f, int& p, int& l) {
    const int pr = (f & 3) | (((f >> 3) & 3) << 2);
    const int c = ((f >> 2) & 1) | ((f >> 5) << 1);
    p = 16 * (c % MB) + pr;
    l = c / MB;
  };
  for (int i = blockIdx.y * blockDim.x + threadIdx.x; i < C::SF + C::FP; i += gridDim.y * blockDim.x) {
    int f, col = -1;
    if (i < C::SF) {
      const int jj = i % 4, lane = (i / 4) % kWave, tile = i / (4 * kWave);
      const int b = tile % C::RB, xw = tile / C::RB;  // xw = CBW mw + x
      const int rho = 16 * b + 4 * (lane / 16) + jj;
      f = (rho & ~31) | (rho & 3) | ((rho << 1) & 24) | ((rho >> 2) & 4);  // the inverse of krow
      col = 16 * xw + lane % 16;
    } else {
      f = i - C::SF;
    }
    int p, l;
    proj_chan(f, p, l);
    if (p >= M) continue;
    float v = 0.0f;
    for (int q = 0; q < a.pieces; ++q) v += pc[(size_t)q * C::STATE + i];
    v *= unscale;
    const int fp = p * L + l;
    float* dst = col >= 0 ? &S[(size_t)fp * DH + col] : &z[fp];
    *dst = a.accumulate ? *dst + v : v;
  }
}

template <typename T, int DH, int L, int MB>
static hipError_t cs_run(const CausalArgs& a, hipStream_t s) {
  if (a.export_S != nullptr) {  // pieces already written by a state launch
    hipLaunchKernelGGL((causal_state_export_kernel<T, DH, L, MB>), dim3(a.heads, 16), dim3(256), 0, s, a);
    return hipGetLastError();
  }
  const int per_head = a.state_out != nullptr ? a.pieces : a.parts;
  if (a.state_out != nullptr)
    hipLaunchKernelGGL((causal_kernel<T, DH, L, MB, true, false>), dim3(a.heads * per_head), dim3(512), 0, s, a);
  else
    hipLaunchKernelGGL((causal_kernel<T, DH, L, MB, false, false>), dim3(a.heads * per_head), dim3(512), 0, s, a);
  return hipGetLastError();
}

// features given: FP bf16 features per token in a.phiq, a.phik
template <int DH, int FP>
static hipError_t cs_run_given(const CausalArgs& a, hipStream_t s) {
  const int per_head = a.state_out != nullptr ? a.pieces : a.parts;
  if (a.state_out != nullptr)
    hipLaunchKernelGGL((causal_kernel<__bf16, DH, 1, FP / 16, true, true>), dim3(a.heads * per_head), dim3(512), 0,
                       s, a);
  else
    hipLaunchKernelGGL((causal_kernel<__bf16, DH, 1, FP / 16, false, true>), dim3(a.heads * per_head), dim3(512), 0,
                       s, a);
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

size_t causal_state_floats(Dt dt, int d, int L, int M) {
  const int MB = (M + 15) / 16;
#define X(T_, D_, L_, MB_) \
  if (dt == cs_dt_of<T_>() && d == D_ && L == L_ && MB == MB_) return CsCfg<T_, D_, L_, MB_>::STATE;
  LUNA_CS_CASES(X)
#undef X
  return 0;
}

// (d, features) combinations built with the features given (bf16)
#define LUNA_CS_GIVEN_CASES(X) \
  X(128, 256)                  \
  X(64, 128)

bool causal_given_supported(Dt dt, int d, int D) {
#define X(D_, F_) \
  if (dt == Dt::BF16 && d == D_ && D == F_) return true;
  LUNA_CS_GIVEN_CASES(X)
#undef X
  return false;
}

size_t causal_given_state_floats(int d, int D) {
#define X(D_, F_) \
  if (d == D_ && D == F_) return CsCfg<__bf16, D_, 1, F_ / 16, true>::STATE;
  LUNA_CS_GIVEN_CASES(X)
#undef X
  return 0;
}

hipError_t launch_causal_given(int d, int D, const CausalArgs& a, hipStream_t s) {
#define X(D_, F_) \
  if (d == D_ && D == F_) return cs_run_given<D_, F_>(a, s);
  LUNA_CS_GIVEN_CASES(X)
#undef X
  return hipErrorInvalidValue;
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
