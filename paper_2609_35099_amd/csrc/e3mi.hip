// e3mi: channelwise Clebsch-Gordan tensor product and message-passing
// convolution for MI355X (gfx950).  Kernels and the C ABI declared in
// include/e3mi.h.
//
// Execution model (the same for every kernel that touches features):
//   * lanes = channels.  A 64-lane wave covers C channels with CPL = C/64
//     consecutive channels per lane, so every feature row (C floats) is one
//     coalesced vector load or store; the feature axis is walked in registers.
//   * per edge (or tensor-product row), the channel-independent
//     pre-contraction A[(path, M), m1] = sum_m2 C[M, m1, m2] y[m2] (records
//     grouped by output then x coordinate, App. E.4's MessageTile grouping) is
//     computed once with lane = edge and staged in LDS; the per-channel loop
//     reads it back as wave-uniform broadcasts.  The coupling constants are
//     compile-time literals (generated per irreps variant).
//   * a wave owns one receiver and one group of paths (forward) or one group
//     of whole x blocks (backward); its accumulators live in registers and are
//     stored once (App. E.3 receiver-stationary aggregation).  No atomics.
//   * workgroups are single waves; block ids are mapped so that each XCD
//     walks a contiguous range of receivers and the groups of one receiver run
//     back to back on the same XCD (shared L2 for the sender gathers).
#include <hip/hip_runtime.h>
#include <hipcub/hipcub.hpp>

#include <algorithm>
#include <array>
#include <cstdint>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <type_traits>
#include <vector>

#include "../../include/e3mi.h"
#include "builder.h"
// Forward sweep: 1 keeps the per-edge pre-contraction reads from LDS where
// the generated code requests them, four float4s ahead of their use, with
// scheduling barriers (5.10 -> 5.02 ms; left to the scheduler, each read
// was issued a few instructions before its use).
#ifndef E3_FWD_ALOAD_PIN
#define E3_FWD_ALOAD_PIN 1
#endif
#if E3_FWD_ALOAD_PIN
#define E3_FWD_PIN() __builtin_amdgcn_sched_barrier(0)
#else
#define E3_FWD_PIN() ((void)0)
#endif
// Convolution backward sweep: the A reads of each path, and two float4s
// beyond, requested before the path's code and held there (12.24 -> 12.13
// ms).  The fused-radial backward measured 1% slower with it and the tensor
// product backward keeps the compiler's placement.
#ifndef E3_BWD_ALOAD_PIN
#define E3_BWD_ALOAD_PIN 1
#endif
#include "generated/variants.inc"

namespace {

thread_local std::string g_last_error;

// ------------------------------------------------------------ launch timing
// When enabled, every kernel launch of the library is bracketed by two HIP
// events recorded on the caller's stream; e3_timing_read() resolves them into
// per-kernel summed durations.  Off by default (no events recorded).
struct Timing {
  std::mutex mu;
  bool on = false;
  struct Pending {
    std::string name;
    hipEvent_t a, b;
  };
  std::vector<Pending> pending;
  std::vector<hipEvent_t> pool;
  std::map<std::string, std::pair<double, int64_t>> acc;
  hipEvent_t get() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
};
Timing g_timing;

struct TimedLaunch {
  hipEvent_t a = nullptr, b = nullptr;
  const char* name;
  hipStream_t st;
  TimedLaunch(const char* n, hipStream_t s) : name(n), st(s) {
    std::lock_guard<std::mutex> lk(g_timing.mu);
    if (!g_timing.on) return;
    a = g_timing.get();
    b = g_timing.get();
    if (a && b && hipEventRecord(a, st) != hipSuccess) a = nullptr;
  }
  ~TimedLaunch() {
    if (!a || !b) return;
    if (hipEventRecord(b, st) != hipSuccess) return;
    std::lock_guard<std::mutex> lk(g_timing.mu);
    g_timing.pending.push_back({name, a, b});
  }
};

#define E3_HIP(call)                                                          \
  do {                                                                        \
    hipError_t err_ = (call);                                                 \
    if (err_ != hipSuccess) {                                                 \
      g_last_error = std::string(#call) + ": " + hipGetErrorString(err_);     \
      return E3_ERR_HIP;                                                      \
    }                                                                         \
  } while (0)

constexpr int kWave = 64;
constexpr int kXcd = 8;

// Row-tile kernels (tensor product, its backward, the record path): block ->
// (tile, part).  With XCD, the `per` parts (groups, channel slabs) of tile T
// run on XCD T % 8 in consecutive dispatch rounds, so that the parts of one
// row, which read the neighbouring pieces of its rows, run on one XCD
// together; otherwise the parts of a tile are consecutive blocks.  The grid
// is tile_grid(...) blocks; blocks past the last tile return false.
#ifndef E3_TP_XCD
#define E3_TP_XCD 1
#endif
template <bool XCD>
__device__ __forceinline__ bool tile_of(int64_t rows, int rows_per_tile, int per, int64_t& tile, int& part) {
  const int64_t ntiles = (rows + rows_per_tile - 1) / rows_per_tile;
  if constexpr (XCD) {
    const int64_t u = blockIdx.x / kXcd;
    part = (int)(u % per);
    tile = (u / per) * kXcd + blockIdx.x % kXcd;
  } else {
    part = (int)(blockIdx.x % per);
    tile = blockIdx.x / per;
  }
  return tile < ntiles;
}
inline int64_t tile_grid(bool xcd, int64_t rows, int rows_per_tile, int per) {
  const int64_t ntiles = (rows + rows_per_tile - 1) / rows_per_tile;
  return (xcd ? (ntiles + kXcd - 1) / kXcd * kXcd : ntiles) * per;
}

// Build-time tuning knobs: minimum resident waves per SIMD requested from the
// compiler for the forward and backward sweeps, and channels per lane of the
// backward sweep when C > 64.
#ifndef E3_FWD_MIN_WAVES
#define E3_FWD_MIN_WAVES 2
#endif
#ifndef E3_BWD_MIN_WAVES
#define E3_BWD_MIN_WAVES 2
#endif
#ifndef E3_BWD_CPL
#define E3_BWD_CPL 1
#endif
#ifndef E3_FWD_CPL
#define E3_FWD_CPL 2
#endif
#ifndef E3_DX_VEC
#define E3_DX_VEC 8
#endif
#ifndef E3_DX_UNROLL
#define E3_DX_UNROLL 2
#endif
#define E3_PRAGMA(x) _Pragma(#x)
#define E3_UNROLL(n) E3_PRAGMA(unroll n)
#ifndef E3_FWD_PREFETCH3
#define E3_FWD_PREFETCH3 1
#endif
#ifndef E3_RAD_WREG
#define E3_RAD_WREG 1
#endif
// 1: the backward sweep double-buffers the path weights as well as the x rows.
#ifndef E3_BWD_DB_S
#define E3_BWD_DB_S 1
#endif
// Cache policy of the backward sweeps' x-cotangent partials: non-temporal (2).
// Plain stores measured slower in both the sweep and the segment sum that
// reads them back (12.67 against 12.35 ms and 1.94 against 1.84 ms).
#ifndef E3_T_STORE_AUX
#define E3_T_STORE_AUX 2
#endif
constexpr int kMaxChannels = 1024;

typedef float f2v __attribute__((ext_vector_type(2)));
typedef float f4v __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------ row load/store
template <int CPL>
__device__ __forceinline__ void ld_row(const float* __restrict__ p, float (&v)[CPL]) {
  if constexpr (CPL == 1) {
    v[0] = *p;
  } else if constexpr (CPL == 2) {
    f2v t = *reinterpret_cast<const f2v*>(p);
    v[0] = t.x, v[1] = t.y;
  } else {
    f4v t = *reinterpret_cast<const f4v*>(p);
    v[0] = t.x, v[1] = t.y, v[2] = t.z, v[3] = t.w;
  }
}

// streamed once: non-temporal (does not displace the gathered node features)
template <int CPL>
__device__ __forceinline__ void ld_row_nt(const float* __restrict__ p, float (&v)[CPL]) {
  if constexpr (CPL == 1) {
    v[0] = __builtin_nontemporal_load(p);
  } else if constexpr (CPL == 2) {
    f2v t = __builtin_nontemporal_load(reinterpret_cast<const f2v*>(p));
    v[0] = t.x, v[1] = t.y;
  } else {
    f4v t = __builtin_nontemporal_load(reinterpret_cast<const f4v*>(p));
    v[0] = t.x, v[1] = t.y, v[2] = t.z, v[3] = t.w;
  }
}

template <int CPL>
__device__ __forceinline__ void st_row_nt(float* __restrict__ p, const float (&v)[CPL]) {
  if constexpr (CPL == 1) {
    __builtin_nontemporal_store(v[0], p);
  } else if constexpr (CPL == 2) {
    f2v t = {v[0], v[1]};
    __builtin_nontemporal_store(t, reinterpret_cast<f2v*>(p));
  } else {
    f4v t = {v[0], v[1], v[2], v[3]};
    __builtin_nontemporal_store(t, reinterpret_cast<f4v*>(p));
  }
}

template <int CPL>
__device__ __forceinline__ void st_row(float* __restrict__ p, const float (&v)[CPL]) {
  if constexpr (CPL == 1) {
    *p = v[0];
  } else if constexpr (CPL == 2) {
    *reinterpret_cast<f2v*>(p) = f2v{v[0], v[1]};
  } else {
    *reinterpret_cast<f4v*>(p) = f4v{v[0], v[1], v[2], v[3]};
  }
}

// Rows of C floats addressed through a buffer resource: a wave-uniform base
// (one edge's or one node's block of rows), a per-lane byte offset (the lane's
// channels) and a per-row scalar offset, so no per-row vector address math.
// Offsets outside the block read as zero and stores there are dropped.
struct RowBuf {
  __amdgpu_buffer_rsrc_t r;
  int voff;      // lane's first channel, bytes
  int rowbytes;  // C * 4
};

__device__ __forceinline__ RowBuf row_buf(const float* base, int64_t nbytes, int q, int C) {
  RowBuf b;
  b.r = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), (short)0,
                                          (int)(nbytes < 0x7fffffff ? nbytes : 0x7fffffff), 0x00020000);
  b.voff = q * 4;
  b.rowbytes = C * 4;
  return b;
}

// Read-only tables (records, job lists) through the constant address space,
// so that uniform reads become scalar loads.
template <class T>
using ConstPtr = const __attribute__((address_space(4))) T*;

constexpr int kNT = 2;  // non-temporal loads of data streamed once
// Stores of streamed outputs: non-temporal.  A pure write stream runs faster
// with plain stores on MI355X, but in these mixed read/write kernels plain
// stores were measured equal or slower (TP forward equal, TP backward 3.85 ms
// against 3.43 ms, convolution step 21.3 ms against 20.8 ms).
#ifndef E3_STORE_AUX
#define E3_STORE_AUX 2
#endif
constexpr int kST = E3_STORE_AUX;

template <int CPL, int AUX = 0>
__device__ __forceinline__ void bld(const RowBuf& b, int row, float (&v)[CPL]) {
  const int so = row * b.rowbytes;
  if constexpr (CPL == 1) {
    v[0] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(b.r, b.voff, so, AUX));
  } else if constexpr (CPL == 2) {
    f2v t = __builtin_bit_cast(f2v, __builtin_amdgcn_raw_buffer_load_b64(b.r, b.voff, so, AUX));
    v[0] = t.x, v[1] = t.y;
  } else {
    f4v t = __builtin_bit_cast(f4v, __builtin_amdgcn_raw_buffer_load_b128(b.r, b.voff, so, AUX));
    v[0] = t.x, v[1] = t.y, v[2] = t.z, v[3] = t.w;
  }
}

template <int CPL, int AUX = 0>
__device__ __forceinline__ void bst(const RowBuf& b, int row, const float (&v)[CPL]) {
  const int so = row * b.rowbytes;
  if constexpr (CPL == 1) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v[0]), b.r, b.voff, so, AUX);
  } else if constexpr (CPL == 2) {
    typedef unsigned u2v __attribute__((ext_vector_type(2)));
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u2v, f2v{v[0], v[1]}), b.r, b.voff, so, AUX);
  } else {
    typedef unsigned u4v __attribute__((ext_vector_type(4)));
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u4v, f4v{v[0], v[1], v[2], v[3]}), b.r, b.voff, so,
                                           AUX);
  }
}

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ int imin(int a, int b) { return a < b ? a : b; }

// First channel and active lanes of a slab.
template <int CPL>
__device__ __forceinline__ void slab_of(int C, int sl, int& ch0, int& lanes) {
  ch0 = sl * kWave * CPL;
  lanes = imin(kWave, (C - ch0) / CPL);
}

// Unit vector of an edge; a zero vector maps to 0 (then Y_0 = 1, all else 0).
__device__ __forceinline__ void unit_of(const float* __restrict__ vec, int64_t e, float& ux, float& uy,
                                        float& uz, float& inv) {
  const float vx = vec[3 * e], vy = vec[3 * e + 1], vz = vec[3 * e + 2];
  const float r2 = vx * vx + vy * vy + vz * vz;
  inv = r2 > 0.0f ? rsqrtf(r2) : 0.0f;
  ux = vx * inv, uy = vy * inv, uz = vz * inv;
}

// Lane exchanges of gfx950 behind the wave reductions.  swap32(a, b) leaves
// a = [a of lanes 0..31, b of lanes 0..31] and b = [a of lanes 32..63, b of
// lanes 32..63]; swap16 does the same between the odd 16-lane rows of a and
// the even rows of b, within each half.  dpp<CTRL>(v) reads v of another lane
// of the same 16-lane row (quad permutes, rotate by 8 = lane ^ 8, mirror of
// each 8-lane half = lane ^ 7).
__device__ __forceinline__ void swap32(float& a, float& b) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b), false, false);
  a = __uint_as_float(r[0]), b = __uint_as_float(r[1]);
}
__device__ __forceinline__ void swap16(float& a, float& b) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false, false);
  a = __uint_as_float(r[0]), b = __uint_as_float(r[1]);
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppXor8 = 0x128, kDppXor7 = 0x141;
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, true));
}

// Sum of v[16] over the 64 lanes of the wave by a fixed tree (transposed
// halving: each stage keeps half of the values and exchanges the other half,
// on lane bits 5, 4, 3, then 2 paired by the half-row mirror, then a quad
// sum; bk below is bit k of the lane); lane l ends with the total of index
// l / 4.
__device__ __forceinline__ float wave_reduce16(const float (&v)[16], int lane) {
  float w8[8], w4[4], w2[2];
  const bool b3 = lane & 8, b2 = lane & 4;
#pragma unroll
  for (int i = 0; i < 8; ++i) {  // index i + 8 b5, summed over lane bit 5
    float a = v[i], b = v[i + 8];
    swap32(a, b);
    w8[i] = a + b;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {  // index i + 4 b4 + 8 b5, summed over bits 4, 5
    float a = w8[i], b = w8[i + 4];
    swap16(a, b);
    w4[i] = a + b;
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {  // index i + 2 b3 + 4 b4 + 8 b5, summed over bits 3..5
    const float send = b3 ? w4[i] : w4[i + 2];
    const float keep = b3 ? w4[i + 2] : w4[i];
    w2[i] = keep + dpp<kDppXor8>(send);
  }
  // index l / 4; the partner l ^ 7 has the same bits 3..5 and the other bit 2,
  // and the quad sum then covers all eight values of the low three bits
  float w1 = (b2 ? w2[1] : w2[0]) + dpp<kDppXor7>(b2 ? w2[0] : w2[1]);
  w1 += dpp<kDppXor1>(w1);
  w1 += dpp<kDppXor2>(w1);
  return w1;
}

// ------------------------------------------------------------ harmonics
template <int L>
__device__ __forceinline__ void sh_of(float x, float y, float z, float* Y) {
  if constexpr (L == 0) e3gen::sh_l0(x, y, z, Y);
  else if constexpr (L == 1) e3gen::sh_l1(x, y, z, Y);
  else if constexpr (L == 2) e3gen::sh_l2(x, y, z, Y);
  else e3gen::sh_l3(x, y, z, Y);
}
template <int L>
__device__ __forceinline__ void sh_grad_of(float x, float y, float z, const float* dY, float& gx, float& gy,
                                           float& gz) {
  if constexpr (L == 0) e3gen::sh_grad_l0(x, y, z, dY, gx, gy, gz);
  else if constexpr (L == 1) e3gen::sh_grad_l1(x, y, z, dY, gx, gy, gz);
  else if constexpr (L == 2) e3gen::sh_grad_l2(x, y, z, dY, gx, gy, gz);
  else e3gen::sh_grad_l3(x, y, z, dY, gx, gy, gz);
}

// dvec = (I - u u^T) g / |r| with g the gradient of the harmonic polynomials.
__device__ __forceinline__ void project(float ux, float uy, float uz, float inv, float gx, float gy, float gz,
                                        float& dx, float& dy, float& dz) {
  const float ug = ux * gx + uy * gy + uz * gz;
  dx = (gx - ux * ug) * inv;
  dy = (gy - uy * ug) * inv;
  dz = (gz - uz * ug) * inv;
}

template <int L>
__global__ __launch_bounds__(256) void k_sh(const float* __restrict__ vec, float* __restrict__ y, int64_t n) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= n) return;
  float ux, uy, uz, inv;
  unit_of(vec, e, ux, uy, uz, inv);
  constexpr int D = (L + 1) * (L + 1);
  float Y[D];
  sh_of<L>(ux, uy, uz, Y);
#pragma unroll
  for (int i = 0; i < D; ++i) y[e * D + i] = Y[i];
}

template <int L>
__global__ __launch_bounds__(256) void k_sh_bwd(const float* __restrict__ vec, const float* __restrict__ dy,
                                                float* __restrict__ dvec, int64_t n) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= n) return;
  float ux, uy, uz, inv;
  unit_of(vec, e, ux, uy, uz, inv);
  constexpr int D = (L + 1) * (L + 1);
  float dY[D];
#pragma unroll
  for (int i = 0; i < D; ++i) dY[i] = dy[e * D + i];
  float gx, gy, gz, ox, oy, oz;
  sh_grad_of<L>(ux, uy, uz, dY, gx, gy, gz);
  project(ux, uy, uz, inv, gx, gy, gz, ox, oy, oz);
  dvec[3 * e] = ox, dvec[3 * e + 1] = oy, dvec[3 * e + 2] = oz;
}

// ------------------------------------------------------------ tensor product
constexpr int kTpRows = 8;  // rows whose pre-contraction is staged per LDS batch

template <class V, int CPL>
__global__ __launch_bounds__(kWave) void k_tp(const float* __restrict__ x, const float* __restrict__ y,
                                              const float* __restrict__ w, float* __restrict__ z, int64_t rows,
                                              int C, int nslab) {
  using T = typename V::TP;
  __shared__ f4v smem[(kTpRows * T::NA + 3) / 4];
  float* sA = reinterpret_cast<float*>(smem);
  const int lane = threadIdx.x;
  int sl;
  int64_t tile;
  if (!tile_of<false>(rows, kTpRows, nslab, tile, sl)) return;
  int ch0, lanes;
  slab_of<CPL>(C, sl, ch0, lanes);
  const int64_t r0 = tile * kTpRows;
  const int n = (int)((rows - r0) < kTpRows ? (rows - r0) : kTpRows);
  if (lane < n) {
    float Y[V::D_SH];
#pragma unroll
    for (int i = 0; i < V::D_SH; ++i) Y[i] = y[(r0 + lane) * V::D_SH + i];
    T::make_A(Y, sA + lane * T::NA);
  }
  __syncthreads();
  if (lane >= lanes) return;
  const int q = ch0 + lane * CPL;
  for (int j = 0; j < n; ++j) {
    const int64_t r = r0 + j;
    float xv[T::NXR][CPL], wv[T::NPATH][CPL];
    const RowBuf xb = row_buf(x + r * V::D_IN * C, (int64_t)V::D_IN * C * 4, q, C);
    const RowBuf wb = row_buf(w + r * V::NP * C, (int64_t)V::NP * C * 4, q, C);
    const RowBuf zb = row_buf(z + r * V::D_OUT * C, (int64_t)V::D_OUT * C * 4, q, C);
#pragma unroll
    for (int i = 0; i < T::NXR; ++i) bld<CPL, kNT>(xb, T::XROW[i], xv[i]);
#pragma unroll
    for (int i = 0; i < T::NPATH; ++i) bld<CPL, kNT>(wb, T::PATH[i], wv[i]);
    auto st = [&](int row, const float (&v)[CPL]) { bst<CPL, kST>(zb, row, v); };
    T::template rows<CPL>(sA + j * T::NA, xv, wv, st);
  }
}

// ------------------------------------------------------------ tensor product backward
// One wave per (tile of kTpRows rows, group of whole x blocks, channel slab):
// the backward group code of the convolution with the row's dz in place of the
// receiver cotangent; dx and dw rows are stored directly, dy (summed over the
// wave's channels) goes to a per-wave slot that k_tp_bwd_dy adds up.
struct TpbArgs {
  const float* x;
  const float* y;
  const float* w;
  const float* dz;
  float* dx;
  float* dw;
  float* DY;  // [rows, NBG * nslab, 16]
  int64_t rows;
  int C;
  int nslab;
};

template <class V, int G, int CPL>
__device__ __forceinline__ void tpb_task(const TpbArgs& a, int64_t r0, int sl, float* sA, float* sY) {
  using B = typename V::template BG<G>;
  const int lane = threadIdx.x;
  int ch0, lanes;
  slab_of<CPL>(a.C, sl, ch0, lanes);
  const bool act = lane < lanes;
  const int C = a.C, q = ch0 + lane * CPL;
  const int n = (int)((a.rows - r0) < kTpRows ? (a.rows - r0) : kTpRows);
  if (lane < n) {
    float Y[V::D_SH];
#pragma unroll
    for (int i = 0; i < V::D_SH; ++i) Y[i] = a.y[(r0 + lane) * V::D_SH + i];
#pragma unroll
    for (int i = 0; i < V::D_SH; ++i) sY[lane * V::D_SH + i] = Y[i];
    B::make_A(Y, sA + lane * B::NA);
  }
  __syncthreads();
  for (int j = 0; j < n; ++j) {
    const int64_t r = r0 + j;
    float dy[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) dy[i] = 0.0f;
    if (act) {
      const RowBuf xb = row_buf(a.x + r * V::D_IN * C, (int64_t)V::D_IN * C * 4, q, C);
      const RowBuf wb = row_buf(a.w + r * V::NP * C, (int64_t)V::NP * C * 4, q, C);
      const RowBuf zb = row_buf(a.dz + r * V::D_OUT * C, (int64_t)V::D_OUT * C * 4, q, C);
      float xv[B::NXR][CPL], wv[B::NPATH][CPL], dzv[B::NROW][CPL], t[B::NXR][CPL], Yv[V::D_SH];
#pragma unroll
      for (int i = 0; i < B::NXR; ++i) {
        bld<CPL, kNT>(xb, B::XROW[i], xv[i]);
#pragma unroll
        for (int c = 0; c < CPL; ++c) t[i][c] = 0.0f;
      }
#pragma unroll
      for (int i = 0; i < B::NPATH; ++i) bld<CPL, kNT>(wb, B::PATH[i], wv[i]);
#pragma unroll
      for (int i = 0; i < B::NROW; ++i) bld<CPL, kNT>(zb, B::OROW[i], dzv[i]);
#pragma unroll
      for (int i = 0; i < V::D_SH; ++i) Yv[i] = sY[j * V::D_SH + i];
      const RowBuf dwb = row_buf(a.dw + r * V::NP * C, (int64_t)V::NP * C * 4, q, C);
      auto st = [&](int pl, const float (&v)[CPL]) { bst<CPL, kST>(dwb, B::PATH[pl], v); };
      float dyl[V::D_SH];
#pragma unroll
      for (int i = 0; i < V::D_SH; ++i) dyl[i] = 0.0f;
      B::template edge<false, CPL>(sA + j * B::NA, Yv, xv, wv, dzv, t, dyl, st);
#pragma unroll
      for (int i = 0; i < V::D_SH; ++i) dy[i] = dyl[i];
      const RowBuf dxb = row_buf(a.dx + r * V::D_IN * C, (int64_t)V::D_IN * C * 4, q, C);
#pragma unroll
      for (int i = 0; i < B::NXR; ++i) bst<CPL, kST>(dxb, B::XROW[i], t[i]);
    }
    const float tot = wave_reduce16(dy, lane);
    if ((lane & 3) == 0) a.DY[((r * V::NBG + G) * a.nslab + sl) * 16 + (lane >> 2)] = tot;
  }
}

template <class V, int G, int CPL>
__device__ __forceinline__ void tpb_dispatch(const TpbArgs& a, int64_t r0, int g, int sl, float* sA, float* sY) {
  if constexpr (G < V::NBG) {
    if (g == G)
      tpb_task<V, G, CPL>(a, r0, sl, sA, sY);
    else
      tpb_dispatch<V, G + 1, CPL>(a, r0, g, sl, sA, sY);
  }
}

template <class V, int CPL>
__global__ __launch_bounds__(kWave, E3_BWD_MIN_WAVES) void k_tp_bwd(TpbArgs a) {
  __shared__ f4v smem[(kTpRows * (V::MAX_NA_B + V::D_SH) + 3) / 4];
  int t;
  int64_t tile;
  if (!tile_of<E3_TP_XCD>(a.rows, kTpRows, V::NBG * a.nslab, tile, t)) return;
  const int64_t r0 = tile * kTpRows;
  float* sA = reinterpret_cast<float*>(smem);
  tpb_dispatch<V, 0, CPL>(a, r0, t / a.nslab, t % a.nslab, sA, sA + kTpRows * V::MAX_NA_B);
}

// dy[r] = sum over the (group, slab) waves of row r.
template <class V>
__global__ __launch_bounds__(256) void k_tp_bwd_dy(const float* __restrict__ DY, float* __restrict__ dy, int64_t rows,
                                                   int nslab) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= rows) return;
  float acc[V::D_SH];
#pragma unroll
  for (int i = 0; i < V::D_SH; ++i) acc[i] = 0.0f;
  for (int g = 0; g < V::NBG * nslab; ++g)
#pragma unroll
    for (int i = 0; i < V::D_SH; ++i) acc[i] += DY[(r * V::NBG * nslab + g) * 16 + i];
#pragma unroll
  for (int i = 0; i < V::D_SH; ++i) dy[r * V::D_SH + i] = acc[i];
}

// ------------------------------------------------------------ convolution
#ifndef E3_EDGE_BATCH
#define E3_EDGE_BATCH 16
#endif
constexpr int kEdgeBatch = E3_EDGE_BATCH;  // edges whose pre-contraction is staged per LDS batch

struct ConvArgs {
  const float* x;
  const float* vec;
  const float* s;
  const float* dm;
  float* m;
  float* ds;
  float* T;       // backward: per-edge x-cotangent partials, sender-CSR order
  float* DY;      // backward: per-edge, per-group harmonic cotangents
  const int* rowptr;  // receiver CSR
  const int* eid;     // edge id at each receiver-CSR position
  const int* src;     // sender at each receiver-CSR position
  const int* r2s;     // sender-CSR position at each receiver-CSR position
  int n_nodes;
  int chunk;  // receivers per XCD
  int C;
  int nslab;  // channel slabs of 64 lanes x CPL channels
  const float* y;  // harmonics [E, D_sh] given by the caller, or null: from vec
  int accum;       // add to m (forward) / ds (backward) instead of overwriting it
  // backward: bytes of one ds / T row, or 0 when that output is not wanted (the
  // pointer then refers to valid memory that is never written)
  int64_t ds_row, t_row;
  // fused radial weights: s[e, k, q] = sum_j h[e, j] W[j, k, q]
  const float* h;  // [E, K]
  const float* W;  // [K, P, C]
  int K;
  // three-term forward of the double backward: the tangents of x, y and s
  const float* x2;
  const float* y2;
  const float* s2;
};

// Receiver, group and channel slab of this wave: XCD k = blockIdx % 8 walks
// receivers [k*chunk, (k+1)*chunk); the (group, slab) waves of one receiver are
// consecutive on that XCD.
template <int NG>
__device__ __forceinline__ bool task_of(const ConvArgs& a, int& b, int& g, int& sl) {
  const int bid = blockIdx.x;
  const int xcd = bid % kXcd, slot = bid / kXcd;
  const int per = NG * a.nslab;
  const int t = slot % per;
  g = t / a.nslab;
  sl = t % a.nslab;
  const int rl = slot / per;
  b = xcd * a.chunk + rl;
  return rl < a.chunk && b < a.n_nodes;
}


// Harmonics of edge e: from the caller's y when given, else Y(vec_e / |vec_e|).
template <class V>
__device__ __forceinline__ void edge_harmonics(const ConvArgs& a, int64_t e, float (&Y)[V::D_SH]) {
  if (a.y) {
#pragma unroll
    for (int i = 0; i < V::D_SH; ++i) Y[i] = a.y[e * V::D_SH + i];
  } else {
    float ux, uy, uz, inv;
    unit_of(a.vec, e, ux, uy, uz, inv);
    V::sh(ux, uy, uz, Y);
  }
}

template <class V, int G, int CPL, bool ACC>
__device__ __forceinline__ void fwd_task(const ConvArgs& a, int b, int sl, float* sA) {
  using F = typename V::template FG<G>;
  const int lane = threadIdx.x;
  int ch0, lanes;
  slab_of<CPL>(a.C, sl, ch0, lanes);
  const bool act = lane < lanes;
  const int C = a.C, q = ch0 + lane * CPL;
  const int e0 = uniform(a.rowptr[b]), e1 = uniform(a.rowptr[b + 1]);
  float acc[F::NROW][CPL];
#pragma unroll
  for (int i = 0; i < F::NROW; ++i)
#pragma unroll
    for (int c = 0; c < CPL; ++c) acc[i][c] = 0.0f;
  for (int eb = e0; eb < e1; eb += kEdgeBatch) {
    const int n = imin(kEdgeBatch, e1 - eb);
    // lane j < n owns edge eb+j for the batch: indices, harmonics, pre-contraction
    int my_e = 0, my_src = 0;
    if (lane < n) {
      my_e = a.eid[eb + lane];
      my_src = a.src[eb + lane];
      float Y[V::D_SH];
      edge_harmonics<V>(a, my_e, Y);
      F::make_A(Y, sA + lane * F::NA);
    }
    __syncthreads();
    if (act) {
      // two register buffers: the rows of edge j+1 are in flight while edge j computes
      float xa[F::NXR][CPL], sa[F::NPATH][CPL], xb[F::NXR][CPL], sb[F::NPATH][CPL];
      auto load = [&](int j, float (&xv)[F::NXR][CPL], float (&sv)[F::NPATH][CPL]) {
        const int64_t e = __builtin_amdgcn_readlane(my_e, j);
        const int64_t snd = __builtin_amdgcn_readlane(my_src, j);
        const RowBuf xb_ = row_buf(a.x + snd * V::D_IN * C, (int64_t)V::D_IN * C * 4, q, C);
        const RowBuf sb_ = row_buf(a.s + e * V::NP * C, (int64_t)V::NP * C * 4, q, C);
#pragma unroll
        for (int i = 0; i < F::NXR; ++i) bld<CPL>(xb_, F::XROW[i], xv[i]);
#pragma unroll
        for (int i = 0; i < F::NPATH; ++i) bld<CPL, kNT>(sb_, F::PATH[i], sv[i]);
      };
      // a third register buffer where the group's footprint (sums and three
      // x, s buffers) leaves room: above about 220 registers it spilled (the
      // l <= 2 single-group layout, 25% slower than with two buffers)
      if constexpr (E3_FWD_PREFETCH3 && (F::NROW + 3 * (F::NXR + F::NPATH)) * CPL <= 220) {
        // the rows of edges j+1 and j+2 are in flight while j computes
        float xc[F::NXR][CPL], sc[F::NPATH][CPL];
        load(0, xa, sa);
        if (1 < n) load(1, xb, sb);
        for (int j = 0; j < n; j += 3) {
          if (j + 2 < n) load(j + 2, xc, sc);
          F::template edge<CPL>(sA + j * F::NA, xa, sa, acc);
          if (j + 1 < n) {
            if (j + 3 < n) load(j + 3, xa, sa);
            F::template edge<CPL>(sA + (j + 1) * F::NA, xb, sb, acc);
          }
          if (j + 2 < n) {
            if (j + 4 < n) load(j + 4, xb, sb);
            F::template edge<CPL>(sA + (j + 2) * F::NA, xc, sc, acc);
          }
        }
      } else {
        load(0, xa, sa);
        for (int j = 0; j < n; j += 2) {
          if (j + 1 < n) load(j + 1, xb, sb);
          F::template edge<CPL>(sA + j * F::NA, xa, sa, acc);
          if (j + 1 < n) {
            if (j + 2 < n) load(j + 2, xa, sa);
            F::template edge<CPL>(sA + (j + 1) * F::NA, xb, sb, acc);
          }
        }
      }
    }
    __syncthreads();
  }
  if (act) {
    const RowBuf mb = row_buf(a.m + (int64_t)b * V::D_OUT * C, (int64_t)V::D_OUT * C * 4, q, C);
    if constexpr (ACC) {
#pragma unroll
      for (int i = 0; i < F::NROW; ++i) {
        float o[CPL];
        bld<CPL>(mb, F::OROW[i], o);
#pragma unroll
        for (int c = 0; c < CPL; ++c) acc[i][c] += o[c];
      }
    }
#pragma unroll
    for (int i = 0; i < F::NROW; ++i) bst<CPL, kST>(mb, F::OROW[i], acc[i]);
  }
}

template <class V, int G, int CPL, bool ACC>
__device__ __forceinline__ void fwd_dispatch(const ConvArgs& a, int b, int g, int sl, float* sA) {
  if constexpr (G < V::NFG) {
    if (g == G)
      fwd_task<V, G, CPL, ACC>(a, b, sl, sA);
    else
      fwd_dispatch<V, G + 1, CPL, ACC>(a, b, g, sl, sA);
  }
}

// ACC: m += the result (the double backward's sums) instead of m = result.
template <class V, int CPL, bool ACC>
__global__ __launch_bounds__(kWave, E3_FWD_MIN_WAVES) void k_conv_fwd(ConvArgs a) {
  __shared__ f4v smem[(kEdgeBatch * V::MAX_NA_F + 3) / 4];
  int b, g, sl;
  if (!task_of<V::NFG>(a, b, g, sl)) return;
  fwd_dispatch<V, 0, CPL, ACC>(a, b, g, sl, reinterpret_cast<float*>(smem));
}

// The double backward's output cotangent in one pass over the receiver-sorted
// edges (the sum of the three forward products of eq. conv-bwd-bwd-ddm):
//   m[b] = sum_e s_e (A_e x2_src + A2_e x_src) + s2_e (A_e x_src),
// A from the caller's harmonics y, A2 from their tangent y2; one channel per
// lane, smaller edge batches (two pre-contractions per edge share the LDS).
constexpr int kEdgeBatch3 = 8;

template <class V, int G>
__device__ __forceinline__ void fwd3_task(const ConvArgs& a, int b, int sl, float* sA, float* sA2) {
  using F = typename V::template FG<G>;
  const int lane = threadIdx.x;
  int ch0, lanes;
  slab_of<1>(a.C, sl, ch0, lanes);
  const bool act = lane < lanes;
  const int C = a.C, q = ch0 + lane;
  const int e0 = uniform(a.rowptr[b]), e1 = uniform(a.rowptr[b + 1]);
  float acc[F::NROW][1];
#pragma unroll
  for (int i = 0; i < F::NROW; ++i) acc[i][0] = 0.0f;
  for (int eb = e0; eb < e1; eb += kEdgeBatch3) {
    const int n = imin(kEdgeBatch3, e1 - eb);
    int my_e = 0, my_src = 0;
    if (lane < n) {
      my_e = a.eid[eb + lane];
      my_src = a.src[eb + lane];
      float Y[V::D_SH], Yd[V::D_SH];
#pragma unroll
      for (int i = 0; i < V::D_SH; ++i) {
        Y[i] = a.y[(int64_t)my_e * V::D_SH + i];
        Yd[i] = a.y2[(int64_t)my_e * V::D_SH + i];
      }
      F::make_A(Y, sA + lane * F::NA);
      F::make_A(Yd, sA2 + lane * F::NA);
    }
    __syncthreads();
    if (act) {
      float xa[F::NXR][1], xda[F::NXR][1], sa[F::NPATH][1], sda[F::NPATH][1];
      float xb[F::NXR][1], xdb[F::NXR][1], sb[F::NPATH][1], sdb[F::NPATH][1];
      auto load = [&](int j, float (&xv)[F::NXR][1], float (&xdv)[F::NXR][1], float (&sv)[F::NPATH][1],
                      float (&sdv)[F::NPATH][1]) {
        const int64_t e = __builtin_amdgcn_readlane(my_e, j);
        const int64_t snd = __builtin_amdgcn_readlane(my_src, j);
        const RowBuf xr = row_buf(a.x + snd * V::D_IN * C, (int64_t)V::D_IN * C * 4, q, C);
        const RowBuf x2r = row_buf(a.x2 + snd * V::D_IN * C, (int64_t)V::D_IN * C * 4, q, C);
        const RowBuf sr = row_buf(a.s + e * V::NP * C, (int64_t)V::NP * C * 4, q, C);
        const RowBuf s2r = row_buf(a.s2 + e * V::NP * C, (int64_t)V::NP * C * 4, q, C);
#pragma unroll
        for (int i = 0; i < F::NXR; ++i) bld<1>(xr, F::XROW[i], xv[i]), bld<1>(x2r, F::XROW[i], xdv[i]);
#pragma unroll
        for (int i = 0; i < F::NPATH; ++i) bld<1, kNT>(sr, F::PATH[i], sv[i]), bld<1, kNT>(s2r, F::PATH[i], sdv[i]);
      };
      load(0, xa, xda, sa, sda);
      for (int j = 0; j < n; j += 2) {
        if (j + 1 < n) load(j + 1, xb, xdb, sb, sdb);
        F::template edge3<1>(sA + j * F::NA, sA2 + j * F::NA, xa, xda, sa, sda, acc);
        if (j + 1 < n) {
          if (j + 2 < n) load(j + 2, xa, xda, sa, sda);
          F::template edge3<1>(sA + (j + 1) * F::NA, sA2 + (j + 1) * F::NA, xb, xdb, sb, sdb, acc);
        }
      }
    }
    __syncthreads();
  }
  if (act) {
    const RowBuf mb = row_buf(a.m + (int64_t)b * V::D_OUT * C, (int64_t)V::D_OUT * C * 4, q, C);
#pragma unroll
    for (int i = 0; i < F::NROW; ++i) bst<1, kST>(mb, F::OROW[i], acc[i]);
  }
}

template <class V, int G>
__device__ __forceinline__ void fwd3_dispatch(const ConvArgs& a, int b, int g, int sl, float* sA, float* sA2) {
  if constexpr (G < V::NFG) {
    if (g == G)
      fwd3_task<V, G>(a, b, sl, sA, sA2);
    else
      fwd3_dispatch<V, G + 1>(a, b, g, sl, sA, sA2);
  }
}

template <class V>
__global__ __launch_bounds__(kWave, E3_FWD_MIN_WAVES) void k_conv_fwd3(ConvArgs a) {
  __shared__ f4v smem[(2 * kEdgeBatch3 * V::MAX_NA_F + 3) / 4];
  int b, g, sl;
  if (!task_of<V::NFG>(a, b, g, sl)) return;
  float* sA = reinterpret_cast<float*>(smem);
  fwd3_dispatch<V, 0>(a, b, g, sl, sA, sA + kEdgeBatch3 * V::MAX_NA_F);
}

template <class V, int G, int CPL, bool ACC>
__device__ __forceinline__ void bwd_task(const ConvArgs& a, int b, int sl, float* sA, float* sY) {
  using B = typename V::template BG<G>;
  const int lane = threadIdx.x;
  int ch0, lanes;
  slab_of<CPL>(a.C, sl, ch0, lanes);
  const bool act = lane < lanes;
  const int C = a.C, q = ch0 + lane * CPL;
  const int e0 = uniform(a.rowptr[b]), e1 = uniform(a.rowptr[b + 1]);
  if (e0 == e1) return;
  float dmv[B::NROW][CPL];
  if (act) {
    const RowBuf db = row_buf(a.dm + (int64_t)b * V::D_OUT * C, (int64_t)V::D_OUT * C * 4, q, C);
#pragma unroll
    for (int i = 0; i < B::NROW; ++i) bld<CPL>(db, B::OROW[i], dmv[i]);
  }
  for (int eb = e0; eb < e1; eb += kEdgeBatch) {
    const int n = imin(kEdgeBatch, e1 - eb);
    int my_e = 0, my_src = 0, my_slot = 0;
    if (lane < n) {
      my_e = a.eid[eb + lane];
      my_src = a.src[eb + lane];
      my_slot = a.r2s[eb + lane];
      float Y[V::D_SH];
      edge_harmonics<V>(a, my_e, Y);
#pragma unroll
      for (int i = 0; i < V::D_SH; ++i) sY[lane * V::D_SH + i] = Y[i];
      B::make_A(Y, sA + lane * B::NA);
    }
    __syncthreads();
    float xa[B::NXR][CPL], sa[B::NPATH][CPL], xb[B::NXR][CPL];
#if E3_BWD_DB_S
    float sb[B::NPATH][CPL];
#else
    float (&sb)[B::NPATH][CPL] = sa;
#endif
    auto load_x = [&](int j, float (&xv)[B::NXR][CPL]) {
      if (!act) return;
      const int64_t snd = __builtin_amdgcn_readlane(my_src, j);
      const RowBuf xb_ = row_buf(a.x + snd * V::D_IN * C, (int64_t)V::D_IN * C * 4, q, C);
#pragma unroll
      for (int i = 0; i < B::NXR; ++i) bld<CPL>(xb_, B::XROW[i], xv[i]);
    };
    auto load_s = [&](int j, float (&sv)[B::NPATH][CPL]) {
      if (!act) return;
      const int64_t e = __builtin_amdgcn_readlane(my_e, j);
      const RowBuf sb_ = row_buf(a.s + e * V::NP * C, (int64_t)V::NP * C * 4, q, C);
#pragma unroll
      for (int i = 0; i < B::NPATH; ++i) bld<CPL, kNT>(sb_, B::PATH[i], sv[i]);
    };
    auto compute = [&](int j, const float (&xv)[B::NXR][CPL], const float (&sv)[B::NPATH][CPL]) {
      const int64_t e = __builtin_amdgcn_readlane(my_e, j);
      const int64_t slot = __builtin_amdgcn_readlane(my_slot, j);
      float dy[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) dy[i] = 0.0f;
      if (act) {
        float t[B::NXR][CPL], Yv[V::D_SH];
#pragma unroll
        for (int i = 0; i < B::NXR; ++i)
#pragma unroll
          for (int c = 0; c < CPL; ++c) t[i][c] = 0.0f;
#pragma unroll
        for (int i = 0; i < V::D_SH; ++i) Yv[i] = sY[j * V::D_SH + i];
        // an absent output has row size 0: its stores are dropped by the
        // buffer range check, with no branch in the contraction code
        const RowBuf dsb = row_buf(a.ds + e * V::NP * C, a.ds_row, q, C);
        // accumulating: the old ds of this edge is loaded before the contraction
        // starts, so that its latency is hidden behind the arithmetic
        float old[ACC ? B::NPATH : 1][CPL];
        if constexpr (ACC) {
#pragma unroll
          for (int i = 0; i < B::NPATH; ++i) bld<CPL>(dsb, B::PATH[i], old[i]);
        }
        auto st = [&](int pl, const float (&v)[CPL]) {
          if constexpr (ACC) {
            float o[CPL];
#pragma unroll
            for (int c = 0; c < CPL; ++c) o[c] = old[pl][c] + v[c];
            bst<CPL, kST>(dsb, B::PATH[pl], o);
          } else {
            bst<CPL, kST>(dsb, B::PATH[pl], v);
          }
        };
        float dyl[V::D_SH];
#pragma unroll
        for (int i = 0; i < V::D_SH; ++i) dyl[i] = 0.0f;
        B::template edge<E3_BWD_ALOAD_PIN != 0, CPL>(sA + j * B::NA, Yv, xv, sv, dmv, t, dyl, st);
#pragma unroll
        for (int i = 0; i < V::D_SH; ++i) dy[i] = dyl[i];
        {
          const RowBuf Tb = row_buf(a.T + slot * V::D_IN * C, a.t_row, q, C);
#pragma unroll
          for (int i = 0; i < B::NXR; ++i) bst<CPL, E3_T_STORE_AUX>(Tb, B::XROW[i], t[i]);
        }
      }
      const float tot = wave_reduce16(dy, lane);
      if ((lane & 3) == 0) a.DY[(((int64_t)(eb + j) * V::NBG + G) * a.nslab + sl) * 16 + (lane >> 2)] = tot;
    };
    load_x(0, xa);
    if (E3_BWD_DB_S) load_s(0, sa);
    for (int j = 0; j < n; j += 2) {
      if (!E3_BWD_DB_S) load_s(j, sa);
      if (j + 1 < n) {
        load_x(j + 1, xb);
        if (E3_BWD_DB_S) load_s(j + 1, sb);
      }
      compute(j, xa, sa);
      if (j + 1 < n) {
        if (!E3_BWD_DB_S) load_s(j + 1, sb);
        if (j + 2 < n) {
          load_x(j + 2, xa);
          if (E3_BWD_DB_S) load_s(j + 2, sa);
        }
        compute(j + 1, xb, sb);
      }
    }
    __syncthreads();
  }
}

template <class V, int G, int CPL, bool ACC>
__device__ __forceinline__ void bwd_dispatch(const ConvArgs& a, int b, int g, int sl, float* sA, float* sY) {
  if constexpr (G < V::NBG) {
    if (g == G)
      bwd_task<V, G, CPL, ACC>(a, b, sl, sA, sY);
    else
      bwd_dispatch<V, G + 1, CPL, ACC>(a, b, g, sl, sA, sY);
  }
}

// ACC: ds += the result (the double backward's sums) instead of ds = result.
template <class V, int CPL, bool ACC>
__global__ __launch_bounds__(kWave, E3_BWD_MIN_WAVES) void k_conv_bwd_edges(ConvArgs a) {
  __shared__ f4v smem[(kEdgeBatch * (V::MAX_NA_B + V::D_SH) + 3) / 4];
  int b, g, sl;
  if (!task_of<V::NBG>(a, b, g, sl)) return;
  float* sA = reinterpret_cast<float*>(smem);
  bwd_dispatch<V, 0, CPL, ACC>(a, b, g, sl, sA, sA + kEdgeBatch * V::MAX_NA_B);
}

// The double backward's three backward sweeps in one (generated BG::edge3):
// per edge, with the harmonics y and their tangent y2 of the caller, x and its
// tangent x2 (senders), s and its tangent s2 (edges) and dm (receiver), it
// stores gs = ds(x2, y, s) + ds(x, y2, s), the x-cotangent partials of
// (x, y2, s) and (x, y, s2) for the sender segment sum, and the per-wave
// harmonic cotangent partials of (x2, y, s) and (x, y, s2).  One channel per
// lane.
template <class V, int G>
__device__ __forceinline__ void bwd3_task(const ConvArgs& a, int b, int sl, float* sY, float* sY2) {
  using B = typename V::template BG<G>;
  const int lane = threadIdx.x;
  int ch0, lanes;
  slab_of<1>(a.C, sl, ch0, lanes);
  const bool act = lane < lanes;
  const int C = a.C, q = ch0 + lane;
  const int e0 = uniform(a.rowptr[b]), e1 = uniform(a.rowptr[b + 1]);
  if (e0 == e1) return;
  float dmv[B::NROW][1];
  if (act) {
    const RowBuf db = row_buf(a.dm + (int64_t)b * V::D_OUT * C, (int64_t)V::D_OUT * C * 4, q, C);
#pragma unroll
    for (int i = 0; i < B::NROW; ++i) bld<1>(db, B::OROW[i], dmv[i]);
  }
  for (int eb = e0; eb < e1; eb += kEdgeBatch) {
    const int n = imin(kEdgeBatch, e1 - eb);
    int my_e = 0, my_src = 0, my_slot = 0;
    if (lane < n) {
      my_e = a.eid[eb + lane];
      my_src = a.src[eb + lane];
      my_slot = a.r2s[eb + lane];
#pragma unroll
      for (int i = 0; i < V::D_SH; ++i) {
        sY[lane * V::D_SH + i] = a.y[(int64_t)my_e * V::D_SH + i];
        sY2[lane * V::D_SH + i] = a.y2[(int64_t)my_e * V::D_SH + i];
      }
    }
    __syncthreads();
    float xa[B::NXR][1], xda[B::NXR][1], sa[B::NPATH][1], sda[B::NPATH][1];
    float xb[B::NXR][1], xdb[B::NXR][1], sb[B::NPATH][1], sdb[B::NPATH][1];
    auto load = [&](int j, float (&xv)[B::NXR][1], float (&xdv)[B::NXR][1], float (&sv)[B::NPATH][1],
                    float (&sdv)[B::NPATH][1]) {
      if (!act) return;
      const int64_t e = __builtin_amdgcn_readlane(my_e, j);
      const int64_t snd = __builtin_amdgcn_readlane(my_src, j);
      const RowBuf xr = row_buf(a.x + snd * V::D_IN * C, (int64_t)V::D_IN * C * 4, q, C);
      const RowBuf x2r = row_buf(a.x2 + snd * V::D_IN * C, (int64_t)V::D_IN * C * 4, q, C);
      const RowBuf sr = row_buf(a.s + e * V::NP * C, (int64_t)V::NP * C * 4, q, C);
      const RowBuf s2r = row_buf(a.s2 + e * V::NP * C, (int64_t)V::NP * C * 4, q, C);
#pragma unroll
      for (int i = 0; i < B::NXR; ++i) bld<1>(xr, B::XROW[i], xv[i]), bld<1>(x2r, B::XROW[i], xdv[i]);
#pragma unroll
      for (int i = 0; i < B::NPATH; ++i) bld<1, kNT>(sr, B::PATH[i], sv[i]), bld<1, kNT>(s2r, B::PATH[i], sdv[i]);
    };
    auto compute = [&](int j, const float (&xv)[B::NXR][1], const float (&xdv)[B::NXR][1],
                       const float (&sv)[B::NPATH][1], const float (&sdv)[B::NPATH][1]) {
      const int64_t e = __builtin_amdgcn_readlane(my_e, j);
      const int64_t slot = __builtin_amdgcn_readlane(my_slot, j);
      float dy[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) dy[i] = 0.0f;
      if (act) {
        float t[B::NXR][1], Yv[V::D_SH], Y2v[V::D_SH], dyl[V::D_SH];
#pragma unroll
        for (int i = 0; i < B::NXR; ++i) t[i][0] = 0.0f;
#pragma unroll
        for (int i = 0; i < V::D_SH; ++i) Yv[i] = sY[j * V::D_SH + i], Y2v[i] = sY2[j * V::D_SH + i], dyl[i] = 0.0f;
        const RowBuf gsb = row_buf(a.ds + e * V::NP * C, (int64_t)V::NP * C * 4, q, C);
        auto st = [&](int pl, const float (&v)[1]) { bst<1, kST>(gsb, B::PATH[pl], v); };
        B::template edge3<1>(Yv, Y2v, xv, xdv, sv, sdv, dmv, t, dyl, st);
#pragma unroll
        for (int i = 0; i < V::D_SH; ++i) dy[i] = dyl[i];
        const RowBuf Tb = row_buf(a.T + slot * V::D_IN * C, (int64_t)V::D_IN * C * 4, q, C);
#pragma unroll
        for (int i = 0; i < B::NXR; ++i) bst<1, E3_T_STORE_AUX>(Tb, B::XROW[i], t[i]);
      }
      const float tot = wave_reduce16(dy, lane);
      if ((lane & 3) == 0) a.DY[(((int64_t)(eb + j) * V::NBG + G) * a.nslab + sl) * 16 + (lane >> 2)] = tot;
    };
    load(0, xa, xda, sa, sda);
    for (int j = 0; j < n; j += 2) {
      if (j + 1 < n) load(j + 1, xb, xdb, sb, sdb);
      compute(j, xa, xda, sa, sda);
      if (j + 1 < n) {
        if (j + 2 < n) load(j + 2, xa, xda, sa, sda);
        compute(j + 1, xb, xdb, sb, sdb);
      }
    }
    __syncthreads();
  }
}

template <class V, int G>
__device__ __forceinline__ void bwd3_dispatch(const ConvArgs& a, int b, int g, int sl, float* sY, float* sY2) {
  if constexpr (G < V::NBG) {
    if (g == G)
      bwd3_task<V, G>(a, b, sl, sY, sY2);
    else
      bwd3_dispatch<V, G + 1>(a, b, g, sl, sY, sY2);
  }
}

template <class V>
// One wave per SIMD: at two, the l <= 3 sweep spilled 136 bytes per lane and
// ran 26.6 ms against 23.4 ms without the spill.
#ifndef E3_BWD3_MIN_WAVES
#define E3_BWD3_MIN_WAVES 1
#endif
__global__ __launch_bounds__(kWave, E3_BWD3_MIN_WAVES) void k_conv_bwd3(ConvArgs a) {
  __shared__ float smem[2 * kEdgeBatch * V::D_SH];
  int b, g, sl;
  if (!task_of<V::NBG>(a, b, g, sl)) return;
  bwd3_dispatch<V, 0>(a, b, g, sl, smem, smem + kEdgeBatch * V::D_SH);
}

// dx[a] = sum of the partials of a's out-edges, in sender-CSR order.  A
// node's partials are one contiguous block of (out-degree) x D_in x C floats;
// the wave reads each slot's D_in x C floats as float4s (lane l takes float4
// l, l+64, ... of its slab) and keeps kDxVec float4 sums per lane.
constexpr int kDxVec = E3_DX_VEC;

__global__ __launch_bounds__(kWave) void k_conv_bwd_dx(const float* __restrict__ T, float* __restrict__ dx,
                                                       const int* __restrict__ rowptr_s, int n_nodes, int chunk,
                                                       int flat4, int nslab, int accum) {
  const int bid = blockIdx.x;
  const int slot = bid / kXcd, sl = slot % nslab, rl = slot / nslab;
  const int node = (bid % kXcd) * chunk + rl;
  if (rl >= chunk || node >= n_nodes) return;
  const int lane = threadIdx.x;
  const int off = (sl * kWave * kDxVec + lane) * 16;  // bytes
  const int s0 = uniform(rowptr_s[node]), s1 = uniform(rowptr_s[node + 1]);
  typedef unsigned u4v __attribute__((ext_vector_type(4)));
  f4v acc[kDxVec];
#pragma unroll
  for (int k = 0; k < kDxVec; ++k) acc[k] = f4v{0.0f, 0.0f, 0.0f, 0.0f};
  const int64_t slot_bytes = (int64_t)flat4 * 16;
  __amdgpu_buffer_rsrc_t o = __builtin_amdgcn_make_buffer_rsrc(dx + (int64_t)node * flat4 * 4, (short)0,
                                                               (int)slot_bytes, 0x00020000);
  E3_UNROLL(E3_DX_UNROLL)
  for (int t = s0; t < s1; ++t) {
    // out-of-range float4s (past D_in x C) read as zero
    __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(T) + (int64_t)t * flat4 * 4, (short)0, (int)slot_bytes, 0x00020000);
#pragma unroll
    for (int k = 0; k < kDxVec; ++k)
      acc[k] += __builtin_bit_cast(f4v, __builtin_amdgcn_raw_buffer_load_b128(r, off, k * kWave * 16, kNT));
  }
  if (accum) {  // old + this sum, so that accumulating equals adding a separate result
#pragma unroll
    for (int k = 0; k < kDxVec; ++k)
      acc[k] += __builtin_bit_cast(f4v, __builtin_amdgcn_raw_buffer_load_b128(o, off, k * kWave * 16, 0));
  }
#pragma unroll
  for (int k = 0; k < kDxVec; ++k)
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u4v, acc[k]), o, off, k * kWave * 16, kST);
}

// dvec of each live edge from its harmonic cotangent (summed over groups).
template <class V>
__global__ __launch_bounds__(256) void k_conv_bwd_dvec(const float* __restrict__ vec, const float* __restrict__ DY,
                                                       const int* __restrict__ eid, float* __restrict__ dvec,
                                                       int64_t n_live, int nslab) {
  const int64_t pos = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (pos >= n_live) return;
  const int64_t e = eid[pos];
  float dY[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) dY[i] = 0.0f;
  for (int g = 0; g < V::NBG * nslab; ++g)
#pragma unroll
    for (int i = 0; i < V::D_SH; ++i) dY[i] += DY[(pos * V::NBG * nslab + g) * 16 + i];
  float ux, uy, uz, inv;
  unit_of(vec, e, ux, uy, uz, inv);
  float gx, gy, gz, ox, oy, oz;
  V::sh_grad(ux, uy, uz, dY, gx, gy, gz);
  project(ux, uy, uz, inv, gx, gy, gz, ox, oy, oz);
  dvec[3 * e] = ox, dvec[3 * e + 1] = oy, dvec[3 * e + 2] = oz;
}

// Padding edges: zero ds rows and dvec (one block per padding edge).
// Zero the rows of padding edges in up to two per-edge arrays (null: skipped).
__global__ __launch_bounds__(256) void k_zero_pad(const int* __restrict__ pad_eid, int64_t n_pad,
                                                  float* __restrict__ p0, int64_t w0, float* __restrict__ p1,
                                                  int64_t w1) {
  const int64_t i = blockIdx.x;
  if (i >= n_pad) return;
  const int64_t e = pad_eid[i];
  if (p0)
    for (int64_t k = threadIdx.x; k < w0; k += blockDim.x) p0[e * w0 + k] = 0.0f;
  if (p1)
    for (int64_t k = threadIdx.x; k < w1; k += blockDim.x) p1[e * w1 + k] = 0.0f;
}

// dy of each live edge: the sum of its per-(group, slab) partials, in order.
template <class V>
__global__ __launch_bounds__(256) void k_conv_bwd_dy(const float* __restrict__ DY, const int* __restrict__ eid,
                                                     float* __restrict__ dy, int64_t n_live, int nslab, int accum) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t r = i / V::D_SH;
  const int c = (int)(i % V::D_SH);
  if (r >= n_live) return;
  float v = 0.0f;
  for (int g = 0; g < V::NBG * nslab; ++g) v += DY[(r * V::NBG * nslab + g) * 16 + c];
  const int64_t o = (int64_t)eid[r] * V::D_SH + c;
  dy[o] = accum ? dy[o] + v : v;
}


// ------------------------------------------------------------ fused radial weights
// The per-edge weights s_e = h_e W (K radial features times a K x (P C)
// matrix) are formed in the sweep kernels on the matrix cores and never
// stored.  One v_mfma_f32_4x4x1f32 (16 blocks of 4x4, K = 1) takes h[edge i][j]
// from lane 4b + i and W[j][k][channel] from every lane; lane 4b + c then holds
// s[edge i][k][its channel] in accumulator register i, i.e. four edges of the
// lane-per-channel layout the contraction code consumes.  K steps of that per
// path give s for four edges.  Both sweeps use one channel per lane.
constexpr int kRadKMax = 16;

// W held in registers (KR = 8, for K <= 8): wr[j][p] = W[j][path p][channel].
template <class V, int NPATH, int KR>
__device__ __forceinline__ void radial_quad_reg(const float (&wr)[KR][NPATH], const float* sH, int q4,
                                                f4v (&s4)[NPATH]) {
  const int lane = threadIdx.x;
#pragma unroll
  for (int p = 0; p < NPATH; ++p) s4[p] = f4v{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int j = 0; j < KR; ++j) {
    const float hv = sH[(q4 + (lane & 3)) * kRadKMax + j];
#pragma unroll
    for (int p = 0; p < NPATH; ++p) s4[p] = __builtin_amdgcn_mfma_f32_4x4x1f32(hv, wr[j][p], s4[p], 0, 0, 0);
  }
}

template <class V, int NPATH>
__device__ __forceinline__ void radial_quad(const RowBuf& wb, const float* sH, int q4, int K, const int (&path)[NPATH],
                                            f4v (&s4)[NPATH]) {
  const int lane = threadIdx.x;
#pragma unroll
  for (int p = 0; p < NPATH; ++p) s4[p] = f4v{0.0f, 0.0f, 0.0f, 0.0f};
  for (int j = 0; j < K; ++j) {
    const float hv = sH[(q4 + (lane & 3)) * kRadKMax + j];
    float wv[NPATH][1];
#pragma unroll
    for (int p = 0; p < NPATH; ++p) bld<1>(wb, j * V::NP + path[p], wv[p]);
#pragma unroll
    for (int p = 0; p < NPATH; ++p) s4[p] = __builtin_amdgcn_mfma_f32_4x4x1f32(hv, wv[p][0], s4[p], 0, 0, 0);
  }
}

// Lane j < n of the batch stages h of its edge (rows past n read as zero).
__device__ __forceinline__ void stage_h(const ConvArgs& a, int lane, int n, int my_e, float* sH) {
  if (lane < kEdgeBatch)
    for (int j = 0; j < a.K; ++j) sH[lane * kRadKMax + j] = lane < n ? a.h[(int64_t)my_e * a.K + j] : 0.0f;
}

template <class V, int G, int KR0>
__device__ __forceinline__ void fwd_rad_task(const ConvArgs& a, int b, int sl, float* sA, float* sH) {
  using F = typename V::template FG<G>;
  // W stays in registers only where the group's estimated footprint (sums,
  // W, four edges of s, two x buffers) leaves room; otherwise it is re-read
  constexpr int KR = (KR0 > 0 && F::NROW + F::NPATH * (KR0 + 4) + 2 * F::NXR <= 230) ? KR0 : 0;
  const int lane = threadIdx.x;
  int ch0, lanes;
  slab_of<1>(a.C, sl, ch0, lanes);
  const bool act = lane < lanes;
  const int C = a.C, q = ch0 + lane;
  const int e0 = uniform(a.rowptr[b]), e1 = uniform(a.rowptr[b + 1]);
  float acc[F::NROW][1];
#pragma unroll
  for (int i = 0; i < F::NROW; ++i) acc[i][0] = 0.0f;
  const RowBuf wb = row_buf(a.W, (int64_t)a.K * V::NP * C * 4, q, C);
  float wr[KR > 0 ? KR : 1][F::NPATH];
  if constexpr (KR > 0) {
#pragma unroll
    for (int j = 0; j < KR; ++j)
#pragma unroll
      for (int p = 0; p < F::NPATH; ++p) {
        float v[1] = {0.0f};
        if (j < a.K) bld<1>(wb, j * V::NP + F::PATH[p], v);
        wr[j][p] = v[0];
      }
  }
  for (int eb = e0; eb < e1; eb += kEdgeBatch) {
    const int n = imin(kEdgeBatch, e1 - eb);
    int my_e = 0, my_src = 0;
    if (lane < n) {
      my_e = a.eid[eb + lane];
      my_src = a.src[eb + lane];
      float ux, uy, uz, inv;
      unit_of(a.vec, my_e, ux, uy, uz, inv);
      float Y[V::D_SH];
      V::sh(ux, uy, uz, Y);
      F::make_A(Y, sA + lane * F::NA);
    }
    stage_h(a, lane, n, my_e, sH);
    __syncthreads();
    float xa[F::NXR][1], xb[F::NXR][1];
    auto load_x = [&](int j, float (&xv)[F::NXR][1]) {
      if (!act) return;
      const int64_t snd = __builtin_amdgcn_readlane(my_src, j);
      const RowBuf xr = row_buf(a.x + snd * V::D_IN * C, (int64_t)V::D_IN * C * 4, q, C);
#pragma unroll
      for (int i = 0; i < F::NXR; ++i) bld<1>(xr, F::XROW[i], xv[i]);
    };
    load_x(0, xa);
    for (int q4 = 0; q4 < n; q4 += 4) {
      f4v s4[F::NPATH];
      if constexpr (KR > 0)
        radial_quad_reg<V, F::NPATH, (KR > 0 ? KR : 1)>(wr, sH, q4, s4);
      else
        radial_quad<V, F::NPATH>(wb, sH, q4, a.K, F::PATH, s4);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = q4 + i;
        if (j < n) {
          float se[F::NPATH][1];
#pragma unroll
          for (int p = 0; p < F::NPATH; ++p) se[p][0] = s4[p][i];
          if (i & 1) {
            if (j + 1 < n) load_x(j + 1, xa);
            if (act) F::template edge<1>(sA + j * F::NA, xb, se, acc);
          } else {
            if (j + 1 < n) load_x(j + 1, xb);
            if (act) F::template edge<1>(sA + j * F::NA, xa, se, acc);
          }
        }
      }
    }
    __syncthreads();
  }
  if (act) {
    const RowBuf mb = row_buf(a.m + (int64_t)b * V::D_OUT * C, (int64_t)V::D_OUT * C * 4, q, C);
#pragma unroll
    for (int i = 0; i < F::NROW; ++i) bst<1, kST>(mb, F::OROW[i], acc[i]);
  }
}

template <class V, int G, int KR>
__device__ __forceinline__ void fwd_rad_dispatch(const ConvArgs& a, int b, int g, int sl, float* sA, float* sH) {
  if constexpr (G < V::NFG) {
    if (g == G)
      fwd_rad_task<V, G, KR>(a, b, sl, sA, sH);
    else
      fwd_rad_dispatch<V, G + 1, KR>(a, b, g, sl, sA, sH);
  }
}

// KR = 8: W in registers (K <= 8); KR = 0: W re-read from cache per 4 edges.
template <class V, int KR>
__global__ __launch_bounds__(kWave, E3_FWD_MIN_WAVES) void k_conv_fwd_rad(ConvArgs a) {
  __shared__ f4v smem[(kEdgeBatch * (V::MAX_NA_F + kRadKMax) + 3) / 4];
  int b, g, sl;
  if (!task_of<V::NFG>(a, b, g, sl)) return;
  float* sA = reinterpret_cast<float*>(smem);
  fwd_rad_dispatch<V, 0, KR>(a, b, g, sl, sA, sA + kEdgeBatch * V::MAX_NA_F);
}

// Backward sweep with radial weights: as k_conv_bwd_edges, but s comes from
// the matrix cores and ds goes to scratch (row = edge id), where the gradient
// kernel below reads it.
template <class V, int G>
__device__ __forceinline__ void bwd_rad_task(const ConvArgs& a, int b, int sl, float* sA, float* sY, float* sH) {
  using B = typename V::template BG<G>;
  const int lane = threadIdx.x;
  int ch0, lanes;
  slab_of<1>(a.C, sl, ch0, lanes);
  const bool act = lane < lanes;
  const int C = a.C, q = ch0 + lane;
  const int e0 = uniform(a.rowptr[b]), e1 = uniform(a.rowptr[b + 1]);
  if (e0 == e1) return;
  float dmv[B::NROW][1];
  if (act) {
    const RowBuf db = row_buf(a.dm + (int64_t)b * V::D_OUT * C, (int64_t)V::D_OUT * C * 4, q, C);
#pragma unroll
    for (int i = 0; i < B::NROW; ++i) bld<1>(db, B::OROW[i], dmv[i]);
  }
  const RowBuf wb = row_buf(a.W, (int64_t)a.K * V::NP * C * 4, q, C);
  for (int eb = e0; eb < e1; eb += kEdgeBatch) {
    const int n = imin(kEdgeBatch, e1 - eb);
    int my_e = 0, my_src = 0, my_slot = 0;
    if (lane < n) {
      my_e = a.eid[eb + lane];
      my_src = a.src[eb + lane];
      my_slot = a.r2s[eb + lane];
      float ux, uy, uz, inv;
      unit_of(a.vec, my_e, ux, uy, uz, inv);
      float Y[V::D_SH];
      V::sh(ux, uy, uz, Y);
#pragma unroll
      for (int i = 0; i < V::D_SH; ++i) sY[lane * V::D_SH + i] = Y[i];
      B::make_A(Y, sA + lane * B::NA);
    }
    stage_h(a, lane, n, my_e, sH);
    __syncthreads();
    float xa[B::NXR][1], xb[B::NXR][1];
    auto load_x = [&](int j, float (&xv)[B::NXR][1]) {
      if (!act) return;
      const int64_t snd = __builtin_amdgcn_readlane(my_src, j);
      const RowBuf xr = row_buf(a.x + snd * V::D_IN * C, (int64_t)V::D_IN * C * 4, q, C);
#pragma unroll
      for (int i = 0; i < B::NXR; ++i) bld<1>(xr, B::XROW[i], xv[i]);
    };
    auto compute = [&](int j, const float (&xv)[B::NXR][1], const float (&sv)[B::NPATH][1]) {
      const int64_t slot = __builtin_amdgcn_readlane(my_slot, j);
      float dy[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) dy[i] = 0.0f;
      if (act) {
        float t[B::NXR][1], Yv[V::D_SH];
#pragma unroll
        for (int i = 0; i < B::NXR; ++i) t[i][0] = 0.0f;
#pragma unroll
        for (int i = 0; i < V::D_SH; ++i) Yv[i] = sY[j * V::D_SH + i];
        const int64_t e = __builtin_amdgcn_readlane(my_e, j);
        const RowBuf dsb = row_buf(a.ds + e * V::NP * C, (int64_t)V::NP * C * 4, q, C);
        auto st = [&](int pl, const float (&v)[1]) { bst<1, kST>(dsb, B::PATH[pl], v); };
        float dyl[V::D_SH];
#pragma unroll
        for (int i = 0; i < V::D_SH; ++i) dyl[i] = 0.0f;
        B::template edge<false, 1>(sA + j * B::NA, Yv, xv, sv, dmv, t, dyl, st);
#pragma unroll
        for (int i = 0; i < V::D_SH; ++i) dy[i] = dyl[i];
        const RowBuf Tb = row_buf(a.T + slot * V::D_IN * C, (int64_t)V::D_IN * C * 4, q, C);
#pragma unroll
        for (int i = 0; i < B::NXR; ++i) bst<1, E3_T_STORE_AUX>(Tb, B::XROW[i], t[i]);
      }
      const float tot = wave_reduce16(dy, lane);
      if ((lane & 3) == 0) a.DY[(((int64_t)(eb + j) * V::NBG + G) * a.nslab + sl) * 16 + (lane >> 2)] = tot;
    };
    load_x(0, xa);
    for (int q4 = 0; q4 < n; q4 += 4) {
      f4v s4[B::NPATH];
      radial_quad<V, B::NPATH>(wb, sH, q4, a.K, B::PATH, s4);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = q4 + i;
        if (j < n) {
          float se[B::NPATH][1];
#pragma unroll
          for (int p = 0; p < B::NPATH; ++p) se[p][0] = s4[p][i];
          if (i & 1) {
            if (j + 1 < n) load_x(j + 1, xa);
            compute(j, xb, se);
          } else {
            if (j + 1 < n) load_x(j + 1, xb);
            compute(j, xa, se);
          }
        }
      }
    }
    __syncthreads();
  }
}

template <class V, int G>
__device__ __forceinline__ void bwd_rad_dispatch(const ConvArgs& a, int b, int g, int sl, float* sA, float* sY,
                                                 float* sH) {
  if constexpr (G < V::NBG) {
    if (g == G)
      bwd_rad_task<V, G>(a, b, sl, sA, sY, sH);
    else
      bwd_rad_dispatch<V, G + 1>(a, b, g, sl, sA, sY, sH);
  }
}

template <class V>
__global__ __launch_bounds__(kWave, E3_BWD_MIN_WAVES) void k_conv_bwd_rad(ConvArgs a) {
  __shared__ f4v smem[(kEdgeBatch * (V::MAX_NA_B + V::D_SH + kRadKMax) + 3) / 4];
  int b, g, sl;
  if (!task_of<V::NBG>(a, b, g, sl)) return;
  float* sA = reinterpret_cast<float*>(smem);
  float* sY = sA + kEdgeBatch * V::MAX_NA_B;
  bwd_rad_dispatch<V, 0>(a, b, g, sl, sA, sY, sY + kEdgeBatch * V::D_SH);
}

// Sum of v[8] over the wave by the same kind of tree as wave_reduce16
// (exchanges on lane bits 5, 4, 3, then a sum over the low three bits); lane l
// ends with the total of index l / 8.
__device__ __forceinline__ float wave_reduce8(const float (&v)[8], int lane) {
  float w4[4], w2[2];
  const bool b3 = lane & 8;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float a = v[i], b = v[i + 4];
    swap32(a, b);
    w4[i] = a + b;
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    float a = w4[i], b = w4[i + 2];
    swap16(a, b);
    w2[i] = a + b;
  }
  float w1 = (b3 ? w2[1] : w2[0]) + dpp<kDppXor8>(b3 ? w2[0] : w2[1]);
  w1 += dpp<kDppXor1>(w1);
  w1 += dpp<kDppXor2>(w1);
  w1 += dpp<kDppXor7>(w1);
  return w1;
}

// Radial gradients from ds (row = edge id, E rows of PC = P*C floats, padding
// edges' rows zero):
//   dW[j][col] = sum_e h[e][j] ds[e][col]   (split over fixed chunks of rows),
//   dh[e][j]   = sum_col ds[e][col] W[j][col] (split over column slabs).
// One wave per (row chunk, column slab); a slab is kGradF float4s per lane,
// lane l owning float4 columns (kGradF sl + f) 64 + l.  The dW outer products
// run on the matrix cores: h[e][4 kq + i] from lane 4b + i times ds[e][col]
// gives dW[4 kq + i][col] in accumulator register i of the lane owning col.
// Both partial sets are added up afterwards in a fixed order, so the result
// does not depend on scheduling.
#ifndef E3_GRAD_ROWS
#define E3_GRAD_ROWS 4
#endif
#ifndef E3_GRAD_DB
#define E3_GRAD_DB 1
#endif
constexpr int kGradF = 1;
constexpr int kGradRows = E3_GRAD_ROWS;  // rows whose loads are issued together

template <int KQ>
__global__ __launch_bounds__(kWave) void k_rad_grad(const float* __restrict__ DS, const float* __restrict__ h,
                                                    const float* __restrict__ W, float* __restrict__ dWp,
                                                    float* __restrict__ DHp, int64_t n_rows, int PC4, int K,
                                                    int nsl4, int rows_per) {
  static_assert(KQ == 2 || KQ == 4, "K <= 8 or K <= 16");
  constexpr int NV = 4 * KQ;
  const int lane = threadIdx.x;
  const int c = blockIdx.x / nsl4, sl = blockIdx.x % nsl4;
  int col4[kGradF];
#pragma unroll
  for (int f = 0; f < kGradF; ++f) col4[f] = (sl * kGradF + f) * kWave + lane;
  const int64_t r0 = (int64_t)c * rows_per;
  const int64_t r1 = r0 + rows_per < n_rows ? r0 + rows_per : n_rows;
  f4v wv[kGradF][NV];
  {
    const __amdgpu_buffer_rsrc_t wr =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(W), (short)0, K * PC4 * 16, 0x00020000);
#pragma unroll
    for (int f = 0; f < kGradF; ++f)
#pragma unroll
      for (int j = 0; j < NV; ++j)
        wv[f][j] = (j < K && col4[f] < PC4)
                       ? __builtin_bit_cast(f4v, __builtin_amdgcn_raw_buffer_load_b128(wr, col4[f] * 16,
                                                                                        j * PC4 * 16, 0))
                       : f4v{0.0f, 0.0f, 0.0f, 0.0f};
  }
  f4v acc[kGradF][4][KQ];
#pragma unroll
  for (int f = 0; f < kGradF; ++f)
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int k = 0; k < KQ; ++k) acc[f][u][k] = f4v{0.0f, 0.0f, 0.0f, 0.0f};
  // Row loads through descriptors bounded by the row: lanes past the last
  // column slab read zero ds, and j >= K reads zero h.
  auto load_row = [&](int64_t r, f4v(&d)[kGradF], float(&hA)[KQ]) {
    const __amdgpu_buffer_rsrc_t rr =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(DS) + r * PC4 * 4, (short)0, PC4 * 16, 0x00020000);
#pragma unroll
    for (int f = 0; f < kGradF; ++f)
      d[f] = __builtin_bit_cast(f4v, __builtin_amdgcn_raw_buffer_load_b128(rr, col4[f] * 16, 0, kNT));
    const __amdgpu_buffer_rsrc_t hr =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(h) + r * K, (short)0, K * 4, 0x00020000);
#pragma unroll
    for (int k = 0; k < KQ; ++k)
      hA[k] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(hr, (4 * k + (lane & 3)) * 4, 0, 0));
  };
  auto row = [&](int64_t r, const f4v(&d)[kGradF], const float(&hA)[KQ]) {
    float dh[NV];
#pragma unroll
    for (int f = 0; f < kGradF; ++f) {
#pragma unroll
      for (int c4 = 0; c4 < 4; ++c4)
#pragma unroll
        for (int k = 0; k < KQ; ++k)
          acc[f][c4][k] = __builtin_amdgcn_mfma_f32_4x4x1f32(hA[k], d[f][c4], acc[f][c4][k], 0, 0, 0);
#pragma unroll
      for (int j = 0; j < NV; ++j) {
        const float t = d[f][0] * wv[f][j][0] + d[f][1] * wv[f][j][1] + d[f][2] * wv[f][j][2] + d[f][3] * wv[f][j][3];
        dh[j] = f == 0 ? t : dh[j] + t;
      }
    }
    float tot;
    if constexpr (NV == 8)
      tot = wave_reduce8(dh, lane);
    else
      tot = wave_reduce16(dh, lane);
    if ((lane & (kWave / NV - 1)) == 0) DHp[((int64_t)sl * n_rows + r) * NV + lane / (kWave / NV)] = tot;
  };
  int64_t rb = r0;
  if constexpr (E3_GRAD_DB) {
    // two batches of rows in flight: the next batch loads while this one computes
    const int64_t nb = (r1 - r0) / kGradRows;
    f4v dA[kGradRows][kGradF], dB[kGradRows][kGradF];
    float hA[kGradRows][KQ], hB[kGradRows][KQ];
    auto load_batch = [&](int64_t b, f4v(&d)[kGradRows][kGradF], float(&hh)[kGradRows][KQ]) {
#pragma unroll
      for (int u = 0; u < kGradRows; ++u) load_row(r0 + b * kGradRows + u, d[u], hh[u]);
    };
    auto run_batch = [&](int64_t b, const f4v(&d)[kGradRows][kGradF], const float(&hh)[kGradRows][KQ]) {
#pragma unroll
      for (int u = 0; u < kGradRows; ++u) row(r0 + b * kGradRows + u, d[u], hh[u]);
    };
    if (nb > 0) load_batch(0, dA, hA);
    for (int64_t b = 0; b < nb; b += 2) {
      if (b + 1 < nb) load_batch(b + 1, dB, hB);
      run_batch(b, dA, hA);
      if (b + 1 < nb) {
        if (b + 2 < nb) load_batch(b + 2, dA, hA);
        run_batch(b + 1, dB, hB);
      }
    }
    rb = r0 + nb * kGradRows;
  } else {
    for (; rb + kGradRows <= r1; rb += kGradRows) {
      f4v d[kGradRows][kGradF];
      float hA[kGradRows][KQ];
#pragma unroll
      for (int u = 0; u < kGradRows; ++u) load_row(rb + u, d[u], hA[u]);
#pragma unroll
      for (int u = 0; u < kGradRows; ++u) row(rb + u, d[u], hA[u]);
    }
  }
  for (; rb < r1; ++rb) {
    f4v d[kGradF];
    float hA[KQ];
    load_row(rb, d, hA);
    row(rb, d, hA);
  }
  // dWp[c][j][col]: register i of acc[f][c4][k] is j = 4k + i, column 4 col4[f] + c4
  float* out = dWp + (int64_t)c * K * PC4 * 4;
#pragma unroll
  for (int f = 0; f < kGradF; ++f)
    if (col4[f] < PC4)
#pragma unroll
      for (int k = 0; k < KQ; ++k)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int j = 4 * k + i;
          if (j < K) {
            f4v v{acc[f][0][k][i], acc[f][1][k][i], acc[f][2][k][i], acc[f][3][k][i]};
            *reinterpret_cast<f4v*>(out + ((int64_t)j * PC4 + col4[f]) * 4) = v;
          }
        }
}

// dW = sum over row chunks of the partials, in chunk order.
__global__ __launch_bounds__(256) void k_rad_dw_sum(const float* __restrict__ dWp, float* __restrict__ dW,
                                                     int64_t n, int nchunk) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float s = 0.0f;
  for (int c = 0; c < nchunk; ++c) s += dWp[(int64_t)c * n + i];
  dW[i] = s;
}

// dh[e] = sum over column slabs of the partials (laid out [slab][edge][NV]),
// in slab order; one thread per (edge, j).
__global__ __launch_bounds__(256) void k_rad_dh_sum(const float* __restrict__ DHp, float* __restrict__ dh,
                                                     int64_t n_rows, int K, int nsl4, int NV) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t r = i / NV;
  const int j = (int)(i % NV);
  if (r >= n_rows) return;
  float s = 0.0f;
  for (int sl = 0; sl < nsl4; ++sl) s += DHp[((int64_t)sl * n_rows + r) * NV + j];
  if (j < K) dh[r * K + j] = s;
}


// ------------------------------------------------------------ linear mixing
// Dense per-irrep channel mixing on the matrix cores (v_mfma_f32_16x16x4f32,
// fp32 in and out).  A destination block of 2l+1 rows per node receives, for
// each of its sources, src[n, src_row + m, k] B[k, col] summed over k and the
// sources, B[k, col] = W[w_off + k ldk + col ldc].  The forward has one job per
// output block (its sources: the input blocks of the same degree and parity);
// dx has one job per input block (its sources: the output blocks it feeds,
// with W read transposed).
//
// One wave per (job, tile of 32 rows, slab of 64 columns).  Operand layout of
// the 16x16x4 instruction: A[i][kk] from lane i + 16 kk, B[kk][j] from lane
// j + 16 kk, D[4 (l / 16) + r][l % 16] in register r of lane l.  Lane l loads
// one float4 of its row (row l % 16 of a 16-row subtile) at columns
// k0 + 4 (l / 16) .. +3; instruction c then uses component c, so the four kk
// of instruction c are k0 + 4 kk + c, and B is read at the same k.  No
// transpose of the rows is needed.
constexpr int kLinMaxJobs = 64;
constexpr int kLinChunks = 64;  // row chunks of the dW reduction (fixed: deterministic)
#ifndef E3_LIN_RT
#define E3_LIN_RT 4
#endif
constexpr int kLinRT = E3_LIN_RT;  // 16-row subtiles per wave in the gather-GEMM
#ifndef E3_LIN_V4
#define E3_LIN_V4 1
#endif
// Row fetches of the dW kernel in flight while one fetch runs (1 or 2; two
// measured 1.29 -> 1.23 ms).
#ifndef E3_LIN_DW_AHEAD
#define E3_LIN_DW_AHEAD 2
#endif
// 1: the gather-GEMM requests the W operands of the next k step with its A
// rows, instead of at the start of the step that uses them (forward 1.147 ->
// 1.110 ms, dx 1.39 -> 1.356 ms; the A rows two steps ahead as well measured
// no better for the forward and 6% slower for dx).
#ifndef E3_LIN_BPF
#define E3_LIN_BPF 1
#endif

struct LinJob {
  int R, dst_row, src_first, nsrc;
};
struct LinSrc {
  int row, pad;
  int64_t w_off;
};
struct LinPair {  // dW slice: input block row, output block row, W offset
  int R, src_row, dst_row, pad;
  int64_t w_off;
};

struct LinArgs {
  const float* src;
  const float* W;
  float* dst;
  const LinJob* jobs;
  const LinSrc* srcs;
  int64_t n;
  int D_src, C_src, D_dst, C_dst, ldk, ldc, njobs, slabs;
  int first[kLinMaxJobs + 1];
};

// V4 (unit column stride, 16-byte aligned W, C_dst a multiple of 4): lane l
// owns the four consecutive columns col0 + 4 (l % 16) .. +3, so one float4 of
// a W row gives B of all four column blocks, and the results leave as float4s.
template <int RT, bool V4>  // RT subtiles of 16 rows per wave
__global__ __launch_bounds__(kWave) void k_lin_gemm(LinArgs a) {
  const int unit = blockIdx.x;
  int lo = 0, hi = a.njobs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.first[mid] <= unit) lo = mid; else hi = mid - 1;
  }
  const LinJob jb = a.jobs[lo];
  const int u = unit - a.first[lo];
  const int col0 = (u % a.slabs) * kWave;
  const int64_t r0 = (int64_t)(u / a.slabs) * (16 * RT);
  const int64_t NR = a.n * jb.R;
  const int lane = threadIdx.x, g = lane >> 4, li = lane & 15;
  f4v acc[RT][4];
#pragma unroll
  for (int s = 0; s < RT; ++s)
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) acc[s][cb] = f4v{0.0f, 0.0f, 0.0f, 0.0f};
  int64_t abase[RT];
  bool aval[RT];
#pragma unroll
  for (int s = 0; s < RT; ++s) {
    const int64_t r = r0 + 16 * s + li;
    aval[s] = r < NR;
    const int64_t nd = aval[s] ? r / jb.R : 0, m = aval[s] ? r % jb.R : 0;
    abase[s] = (nd * a.D_src + m) * a.C_src + 4 * g;
  }
  if constexpr (V4) {
    // Rows past NR and columns past C_dst load in-bounds data of other rows or
    // read zero; the instruction keeps rows and columns apart and those results
    // are not stored, so no masking is needed.  The A rows of the next
    // (source, k-step) load while this one runs.
    const int colv = col0 + 4 * li;
    const bool cv = colv < a.C_dst;
    const ConstPtr<LinSrc> srcs = (ConstPtr<LinSrc>)a.srcs;
    const int ksteps = a.C_src / 16, nsteps = jb.nsrc * ksteps;
    const int bvoff = ((4 * g) * a.ldk + colv) * 4;
    auto load_a = [&](int i, f4v(&v)[RT]) {
      const int t = i / ksteps;
      const float* sp = a.src + (int64_t)srcs[jb.src_first + t].row * a.C_src + (i - t * ksteps) * 16;
#pragma unroll
      for (int s = 0; s < RT; ++s) v[s] = *reinterpret_cast<const f4v*>(sp + abase[s]);
    };
    auto load_b = [&](int i, f4v(&bq)[4]) {
      const int t = i / ksteps, k0 = (i - t * ksteps) * 16;
      const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<float*>(a.W + srcs[jb.src_first + t].w_off), (short)0, a.C_src * a.C_dst * 4, 0x00020000);
#pragma unroll
      for (int c = 0; c < 4; ++c)
        bq[c] = __builtin_bit_cast(f4v, __builtin_amdgcn_raw_buffer_load_b128(wr, bvoff, (k0 + c) * a.ldk * 4, 0));
    };
    auto mfmas = [&](const f4v(&av)[RT], const f4v(&bq)[4]) {
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int cb = 0; cb < 4; ++cb)
#pragma unroll
          for (int s = 0; s < RT; ++s)
            acc[s][cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s][c], bq[c][cb], acc[s][cb], 0, 0, 0);
    };
    if constexpr (E3_LIN_BPF) {
      // one (source, k-step): the W and A operands of step i + 1 (clamped, so
      // the loads are unconditional and the waits count exactly; loads
      // complete in issue order) are requested, then the 64 instructions run
      // on the operands of step i, requested one step earlier
      auto step = [&](int i, const f4v(&av)[RT], const f4v(&bv)[4], f4v(&an)[RT], f4v(&bn)[4]) {
        const int ni = i + 1 < nsteps ? i + 1 : i;
        load_b(ni, bn);
        load_a(ni, an);
        __builtin_amdgcn_sched_barrier(0);
        mfmas(av, bv);
      };
      f4v a0[RT], a1[RT], b0[4], b1[4];
      if (nsteps > 0) load_b(0, b0), load_a(0, a0);
      for (int i = 0; i < nsteps; i += 2) {
        step(i, a0, b0, a1, b1);
        if (i + 1 < nsteps) step(i + 1, a1, b1, a0, b0);
      }
    } else {
      // one (source, k-step): W (cache-resident) first, then the A rows of step
      // i + 1, then the 64 instructions
      auto step = [&](int i, const f4v(&av)[RT], f4v(&an)[RT]) {
        f4v bq[4];
        load_b(i, bq);
        __builtin_amdgcn_sched_barrier(0);
        load_a(i + 1 < nsteps ? i + 1 : i, an);
        __builtin_amdgcn_sched_barrier(0);
        mfmas(av, bq);
      };
      f4v a0[RT], a1[RT];
      if (nsteps > 0) load_a(0, a0);
      for (int i = 0; i < nsteps; i += 2) {
        step(i, a0, a1);
        if (i + 1 < nsteps) step(i + 1, a1, a0);
      }
    }
    // register r of acc[s][cb] in lane l: row 16 s + 4 (l / 16) + r, column col0 + 4 (l % 16) + cb
    if (!cv) return;
#pragma unroll
    for (int s = 0; s < RT; ++s)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = r0 + 16 * s + 4 * g + r;
        if (row >= NR) continue;
        const int64_t nd = row / jb.R, m = row % jb.R;
        float* dp = a.dst + (nd * a.D_dst + jb.dst_row + m) * a.C_dst;
        *reinterpret_cast<f4v*>(dp + colv) = f4v{acc[s][0][r], acc[s][1][r], acc[s][2][r], acc[s][3][r]};
      }
    return;
  }
  // B[k][col] = W[w_off + k ldk + col ldc]: per-lane part in the vector offset,
  // the k step and column block in the (uniform) scalar offset; columns past
  // C_dst read zero through the range check of a per-source descriptor.
  const int col = col0 + li;
  const int bvoff = ((4 * g) * a.ldk + col * a.ldc) * 4;
  const int ncols_valid = a.C_dst - col0;  // uniform
  for (int t = 0; t < jb.nsrc; ++t) {
    const LinSrc sr = a.srcs[jb.src_first + t];
    const float* sp = a.src + (int64_t)sr.row * a.C_src;
    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(a.W + sr.w_off), (short)0, a.C_src * a.C_dst * 4, 0x00020000);
    for (int k0 = 0; k0 < a.C_src; k0 += 16) {
      f4v av[RT];
#pragma unroll
      for (int s = 0; s < RT; ++s)
        av[s] = aval[s] ? *reinterpret_cast<const f4v*>(sp + abase[s] + k0) : f4v{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int c = 0; c < 4; ++c) {
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) {
          float bv = __builtin_bit_cast(
              float, __builtin_amdgcn_raw_buffer_load_b32(wr, bvoff, ((k0 + c) * a.ldk + 16 * cb * a.ldc) * 4, 0));
          if (16 * cb + li >= ncols_valid) bv = 0.0f;
#pragma unroll
          for (int s = 0; s < RT; ++s)
            acc[s][cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s][c], bv, acc[s][cb], 0, 0, 0);
        }
      }
    }
  }
#pragma unroll
  for (int s = 0; s < RT; ++s)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t row = r0 + 16 * s + 4 * g + r;
      if (row >= NR) continue;
      const int64_t nd = row / jb.R, m = row % jb.R;
      float* dp = a.dst + (nd * a.D_dst + jb.dst_row + m) * a.C_dst;
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
        if (16 * cb + li < ncols_valid) dp[col0 + 16 * cb + li] = acc[s][cb][r];
    }
}

// Wt[pair][j][k] = W[w_off(pair) + k C_out + j]: each dW-sized slice
// transposed, so that dx reads B along rows.
__global__ __launch_bounds__(256) void k_lin_transpose(const float* __restrict__ W, const LinPair* __restrict__ pairs,
                                                        float* __restrict__ Wt, int npairs, int C_in, int C_out) {
  const int64_t per = (int64_t)C_in * C_out;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= per * npairs) return;
  const int p = (int)(i / per);
  const int64_t e = i % per;
  const int j = (int)(e / C_in), k = (int)(e % C_in);
  Wt[i] = W[pairs[p].w_off + (int64_t)k * C_out + j];
}

// dW partials: one wave per (pair, row chunk, 64 x 64 tile of W).  Per four
// rows, lane l loads one float4 of x (columns k-tile + 4 (l % 16) .. +3) and
// one of dout (j-tile + 4 (l % 16) .. +3) of row + l / 16; instruction (a, b)
// takes component a as A and b as B (the 16x16x4 reduction index kk is the
// row), so D[a][b][i][j] accumulates x^T dout at k = k-tile + 4 i + a,
// j = j-tile + 4 j + b.
struct LinDwArgs {
  const float* x;
  const float* dout;
  float* dWp;  // [npairs][kLinChunks][C_in][C_out]
  const LinPair* pairs;
  int64_t n;
  int D_in, C_in, D_out, C_out, ktiles, jtiles;
};

__global__ __launch_bounds__(kWave) void k_lin_dw(LinDwArgs a) {
  const int per = kLinChunks * a.ktiles * a.jtiles;
  const int p = blockIdx.x / per, u = blockIdx.x % per;
  const int chunk = u / (a.ktiles * a.jtiles), kt = (u / a.jtiles) % a.ktiles, jt = u % a.jtiles;
  const LinPair pr = a.pairs[p];
  const int64_t NR = a.n * pr.R;
  const int64_t rpc = ((NR + kLinChunks - 1) / kLinChunks + 15) / 16 * 16;  // rows per chunk, a multiple of 16
  const int64_t rb = chunk * rpc < NR ? chunk * rpc : NR, re = rb + rpc < NR ? rb + rpc : NR;
  const int lane = threadIdx.x, g = lane >> 4, li = lane & 15;
  f4v acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f4v{0.0f, 0.0f, 0.0f, 0.0f};
  const int kc = kt * 64 + 4 * li, jc = jt * 64 + 4 * li;  // multiples of 4; C_in, C_out are of 16
  const bool kv = kc < a.C_in, jv = jc < a.C_out;
  // Lane rows rb + g, rb + g + 4, ...: the (node, m) position steps by four
  // rows without a division.  Columns past C_in / C_out read column 0; their
  // results are not stored.
  const int R = pr.R, dq = 4 / R, dr = 4 % R;
  int64_t row = rb + g;
  int m = (int)(row % R);
  int64_t ox = ((row / R) * a.D_in + pr.src_row + m) * a.C_in + (kv ? kc : 0);
  int64_t od = ((row / R) * a.D_out + pr.dst_row + m) * a.C_out + (jv ? jc : 0);
  const int64_t sx = ((int64_t)dq * a.D_in + dr) * a.C_in, wx = (int64_t)(a.D_in - R) * a.C_in;
  const int64_t sd = ((int64_t)dq * a.D_out + dr) * a.C_out, wd = (int64_t)(a.D_out - R) * a.C_out;
  auto advance = [&]() {
    const bool w = m + dr >= R;
    row += 4;
    m += w ? dr - R : dr;
    ox += w ? sx + wx : sx;
    od += w ? sd + wd : sd;
  };
  auto group = [&](const f4v& xa, const f4v& db) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(xa[i], db[j], acc[i][j], 0, 0, 0);
  };
  // Whole fetches of 16 rows (chunks are sized in multiples of 16 rows, so
  // only the last chunk has a tail): no masking, the next fetch in flight.
  // Every fetch is unconditional so that the waits count exactly; the one
  // past the last whole fetch reads row rb again and is not used.
  constexpr int S = 4;
  const int64_t nf = (re - rb) / (4 * S), rfull = rb + nf * 4 * S;
  const int64_t ox0 = ((rb / R) * a.D_in + pr.src_row + rb % R) * a.C_in + (kv ? kc : 0);
  const int64_t od0 = ((rb / R) * a.D_out + pr.dst_row + rb % R) * a.C_out + (jv ? jc : 0);
  auto fetch = [&](f4v(&xs)[S], f4v(&ds)[S]) {
#pragma unroll
    for (int q = 0; q < S; ++q) {
      const bool ok = row < rfull;
      xs[q] = *reinterpret_cast<const f4v*>(a.x + (ok ? ox : ox0));
      ds[q] = *reinterpret_cast<const f4v*>(a.dout + (ok ? od : od0));
      advance();
    }
  };
  if (nf > 0 && E3_LIN_DW_AHEAD == 2) {
    // two fetches in flight while one runs
    f4v xA[S], dA[S], xB[S], dB[S], xC[S], dC[S];
    fetch(xA, dA);
    fetch(xB, dB);
    for (int64_t f = 0; f < nf; ++f) {
      fetch(xC, dC);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int q = 0; q < S; ++q) group(xA[q], dA[q]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int q = 0; q < S; ++q) xA[q] = xB[q], dA[q] = dB[q], xB[q] = xC[q], dB[q] = dC[q];
    }
    // the state ran two fetches ahead: step back to the first row after the whole fetches
    row = rb + g + nf * 4 * S;
    m = (int)(row % R);
    ox = ((row / R) * a.D_in + pr.src_row + m) * a.C_in + (kv ? kc : 0);
    od = ((row / R) * a.D_out + pr.dst_row + m) * a.C_out + (jv ? jc : 0);
  } else if (nf > 0) {
    f4v xA[S], dA[S], xB[S], dB[S];
    fetch(xA, dA);
    for (int64_t f = 0; f < nf; ++f) {
      fetch(xB, dB);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int q = 0; q < S; ++q) group(xA[q], dA[q]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int q = 0; q < S; ++q) xA[q] = xB[q], dA[q] = dB[q];
    }
    // the state ran one fetch ahead: step back to the first row after the whole fetches
    row = rb + g + nf * 4 * S;
    m = (int)(row % R);
    ox = ((row / R) * a.D_in + pr.src_row + m) * a.C_in + (kv ? kc : 0);
    od = ((row / R) * a.D_out + pr.dst_row + m) * a.C_out + (jv ? jc : 0);
  }
  // the last chunk's tail: four-row groups, rows past re read as zero
  for (int64_t r = rb + nf * 4 * S; r < re; r += 4) {
    const bool ok = row < re;
    const f4v xa = ok ? *reinterpret_cast<const f4v*>(a.x + ox) : f4v{0.0f, 0.0f, 0.0f, 0.0f};
    const f4v db = ok ? *reinterpret_cast<const f4v*>(a.dout + od) : f4v{0.0f, 0.0f, 0.0f, 0.0f};
    group(xa, db);
    advance();
  }
  // register r of acc[a][b] in lane l: k = k-tile + 4 (4 (l / 16) + r) + a, j = j-tile + 4 (l % 16) + b
  float* out = a.dWp + ((int64_t)p * kLinChunks + chunk) * a.C_in * a.C_out;
  if (!jv) return;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int k = kt * 64 + 4 * (4 * g + r) + i;
      if (k >= a.C_in) continue;
      f4v v{acc[i][0][r], acc[i][1][r], acc[i][2][r], acc[i][3][r]};
      *reinterpret_cast<f4v*>(out + (int64_t)k * a.C_out + jc) = v;
    }
}

// dW[w_off(p) + e] = sum over the row chunks of pair p, in chunk order.
__global__ __launch_bounds__(256) void k_lin_dw_sum(const float* __restrict__ dWp, const LinPair* __restrict__ pairs,
                                                     float* __restrict__ dW, int npairs, int64_t per) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)npairs * per) return;
  const int p = (int)(i / per);
  const int64_t e = i % per;
  float s = 0.0f;
  for (int c = 0; c < kLinChunks; ++c) s += dWp[((int64_t)p * kLinChunks + c) * per + e];
  dW[pairs[p].w_off + e] = s;
}


// ------------------------------------------------------------ generic records
// Tensor product with caller-supplied records (App. E.2's unfolded form):
//   out[r, o, q] = sum over the records of segment o of v A[r, a, q] B[r, b, (q)]
// A wave takes RB rows of one 64-channel slab.  The operand rows are staged in
// LDS as [a][row][lane] (so one address serves the RB rows of a record), the
// records and segment offsets are read-only for the launch and come through
// the scalar cache, and each record feeds RB fused multiply-adds.  The
// backward is the same kernel on permuted record tables (eq. tp-bwd); with RED
// the outputs are summed over the channels (a shared y's cotangent): per-slab
// partials in fixed lane order, then k_tpg_sum.
struct TpgRec {
  int a, b;
  float v;
  int pad;
};
struct TpgRec64 {
  int a, b;
  double v;
};
template <class T>
struct TpgArgs {
  const T* A;
  const T* B;
  T* out;
  T* part;  // RED: [rows][nslab][dout]
  const int* seg;
  const typename std::conditional<sizeof(T) == 8, TpgRec64, TpgRec>::type* recs;
  int64_t rows;
  int C, nslab, dA, dB, dout;
};


template <class T>
__device__ __forceinline__ T buf_ld(__amdgpu_buffer_rsrc_t r, int off) {
  if constexpr (sizeof(T) == 8)
    return __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
  else
    return __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}

template <class T, bool BSH, bool RED, int RB>
__global__ __launch_bounds__(kWave) void k_tpg(TpgArgs<T> a) {
  using Rec = typename std::conditional<sizeof(T) == 8, TpgRec64, TpgRec>::type;
  const ConstPtr<Rec> recs = (ConstPtr<Rec>)a.recs;
  const ConstPtr<int> seg = (ConstPtr<int>)a.seg;
  extern __shared__ __align__(16) unsigned char lds_raw[];
  T* lds = reinterpret_cast<T*>(lds_raw);
  int sl;
  int64_t tile;
  if (!tile_of<false>(a.rows, RB, a.nslab, tile, sl)) return;
  const int64_t r0 = tile * RB;
  const int nr = a.rows - r0 < RB ? (int)(a.rows - r0) : RB;
  const int lane = threadIdx.x, q = sl * kWave + lane;
  const bool act = q < a.C;
  T* sA = lds;                                                        // [dA][RB][64]
  T* sB = sA + a.dA * RB * kWave;                                     // BSH: [dB][RB], else [dB][RB][64]
  T* sP = sB + (BSH ? ((a.dB * RB + 3) & ~3) : a.dB * RB * kWave);    // RED: [dout][RB][64]
  // Operand loads through descriptors bounded by the block's rows: rows past
  // the end read zero; lanes past C are zeroed (their sums enter RED's total).
  const __amdgpu_buffer_rsrc_t ar = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<T*>(a.A) + r0 * a.dA * a.C, (short)0, (int)((int64_t)nr * a.dA * a.C * sizeof(T)), 0x00020000);
  const __amdgpu_buffer_rsrc_t br = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<T*>(a.B) + r0 * a.dB * (BSH ? 1 : a.C), (short)0,
      (int)((int64_t)nr * a.dB * (BSH ? 1 : a.C) * sizeof(T)), 0x00020000);
#pragma unroll 8
  for (int i = 0; i < a.dA * RB; ++i) {
    const int ai = i / RB, u = i % RB;
    const T v = buf_ld<T>(ar, (int)(((u * a.dA + ai) * a.C + q) * sizeof(T)));
    sA[i * kWave + lane] = act ? v : T(0);
  }
  if constexpr (BSH) {
    for (int i = lane; i < a.dB * RB; i += kWave) {
      const int bi = i / RB, u = i % RB;
      sB[i] = buf_ld<T>(br, (int)((u * a.dB + bi) * sizeof(T)));
    }
  } else {
#pragma unroll 8
    for (int i = 0; i < a.dB * RB; ++i) {
      const int bi = i / RB, u = i % RB;
      const T v = buf_ld<T>(br, (int)(((u * a.dB + bi) * a.C + q) * sizeof(T)));
      sB[i * kWave + lane] = act ? v : T(0);
    }
  }
  __syncthreads();
  int k = seg[0];
  for (int o = 0; o < a.dout; ++o) {
    const int k1 = seg[o + 1];
    T acc[RB];
#pragma unroll
    for (int u = 0; u < RB; ++u) acc[u] = T(0);
#pragma unroll 2
    for (; k < k1; ++k) {
      const int ra = recs[k].a, rbi = recs[k].b;
      const T rv = T(recs[k].v);
      const T* pa = sA + ra * RB * kWave + lane;
#pragma unroll
      for (int u = 0; u < RB; ++u) {
        const T bv = BSH ? sB[rbi * RB + u] : sB[(rbi * RB + u) * kWave + lane];
        acc[u] = fma(rv * pa[u * kWave], bv, acc[u]);
      }
    }
    if constexpr (RED) {
#pragma unroll
      for (int u = 0; u < RB; ++u) sP[(o * RB + u) * kWave + lane] = acc[u];
    } else if (act) {
#pragma unroll
      for (int u = 0; u < RB; ++u)
        if (u < nr) a.out[((r0 + u) * a.dout + o) * a.C + q] = acc[u];
    }
  }
  if constexpr (RED) {
    __syncthreads();
    for (int i = lane; i < a.dout * RB; i += kWave) {
      const int o = i / RB, u = i % RB;
      if (u >= nr) continue;
      T t = T(0);
      for (int l = 0; l < kWave; ++l) t += sP[i * kWave + l];
      a.part[((r0 + u) * a.nslab + sl) * a.dout + o] = t;
    }
  }
}

template <class T>
__global__ __launch_bounds__(256) void k_tpg_sum(const T* __restrict__ part, T* __restrict__ out, int64_t rows,
                                                  int nslab, int dout) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * dout) return;
  const int64_t r = i / dout;
  const int o = (int)(i % dout);
  T t = T(0);
  for (int sl = 0; sl < nslab; ++sl) t += part[(r * nslab + sl) * dout + o];
  out[i] = t;
}

// ------------------------------------------------------------ graph
__global__ void k_graph_keys(const int32_t* __restrict__ snd, const int32_t* __restrict__ rcv, int64_t n_edges,
                             int32_t n_nodes, int32_t pad, uint32_t* __restrict__ key_r, uint32_t* __restrict__ key_s,
                             int32_t* __restrict__ ids, int* __restrict__ bad) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= n_edges) return;
  const int32_t s = snd[e], r = rcv[e];
  if (s < 0 || s >= n_nodes || r < 0 || r >= n_nodes) *bad = 1;  // every writer stores the same value
  const bool is_pad = pad >= 0 && (s == pad || r == pad);
  key_r[e] = is_pad ? (uint32_t)n_nodes : (uint32_t)r;
  key_s[e] = is_pad ? (uint32_t)n_nodes : (uint32_t)s;
  ids[e] = (int32_t)e;
}

// rowptr[b] = first position with key >= b (binary search; keys sorted).
__global__ void k_graph_rowptr(const uint32_t* __restrict__ keys, int64_t n_edges, int32_t n_nodes,
                               int32_t* __restrict__ rowptr) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b > n_nodes) return;
  int64_t lo = 0, hi = n_edges;
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (keys[mid] < (uint32_t)b)
      lo = mid + 1;
    else
      hi = mid;
  }
  rowptr[b] = (int32_t)lo;
}

__global__ void k_graph_finish(const int32_t* __restrict__ snd, const int32_t* __restrict__ eid_r,
                               const int32_t* __restrict__ eid_s, int64_t n_live, int32_t* __restrict__ src_r,
                               int32_t* __restrict__ pos_s) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_live) return;
  src_r[i] = snd[eid_r[i]];
  pos_s[eid_s[i]] = (int32_t)i;
}

__global__ void k_graph_r2s(const int32_t* __restrict__ eid_r, const int32_t* __restrict__ pos_s, int64_t n_live,
                            int32_t* __restrict__ r2s) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_live) return;
  r2s[i] = pos_s[eid_r[i]];
}

unsigned blocks_for(int64_t n, int t) { return (unsigned)std::max<int64_t>(1, (n + t - 1) / t); }

}  // namespace

// ============================================================ handles
struct e3_plan {
  e3b::Layout lay;
  std::vector<e3b::Record> recs;
  int variant = -1;
  // Channels per lane of the forward / tensor-product / dx kernels (the
  // backward sweep always uses 1) and the number of 64-lane channel slabs.
  int cpl_f = 0, cpl_b = 0, nslab_f = 0, nslab_b = 0;
};

struct e3_graph {
  int64_t n_nodes = 0, n_edges = 0, n_live = 0, n_pad = 0;
  int32_t pad = -1;
  int32_t* rowptr_r = nullptr;  // [N+1]
  int32_t* eid_r = nullptr;     // [E] (live first, then padding edges by id)
  int32_t* src_r = nullptr;     // [n_live]
  int32_t* r2s = nullptr;       // [n_live]
  int32_t* rowptr_s = nullptr;  // [N+1]
  int32_t* eid_s = nullptr;     // [E]
  int32_t* pos_s = nullptr;     // [E] scratch
};

namespace {

size_t align256(size_t n) { return (n + 255) & ~size_t(255); }

struct Ws {
  size_t t_bytes, dy_bytes;
};

template <class V>
Ws bwd_ws(const e3_plan* p, const e3_graph* g) {
  Ws w;
  w.t_bytes = align256((size_t)g->n_live * V::D_IN * p->lay.C * sizeof(float));
  w.dy_bytes = align256((size_t)g->n_live * V::NBG * p->nslab_b * 16 * sizeof(float));
  return w;
}

ConvArgs base_args(const e3_plan* p, const e3_graph* g) {
  ConvArgs a{};
  a.rowptr = g->rowptr_r;
  a.eid = g->eid_r;
  a.src = g->src_r;
  a.r2s = g->r2s;
  a.n_nodes = (int)g->n_nodes;
  a.chunk = (int)((g->n_nodes + kXcd - 1) / kXcd);
  a.C = p->lay.C;
  return a;
}

// One forward convolution.  y: caller's harmonics or null (from vec);
// accum: m += instead of m =.
template <class V, int CPL>
e3_status run_fwd(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* y,
                  const float* s, float* m, int accum, hipStream_t st) {
  ConvArgs a = base_args(p, g);
  a.x = x, a.vec = vec, a.y = y, a.s = s, a.m = m, a.accum = accum;
  a.nslab = p->nslab_f;
  if (g->n_nodes == 0) return E3_OK;
  const unsigned grid = (unsigned)(kXcd * a.chunk * V::NFG * a.nslab);
  {
    TimedLaunch t_("conv_fwd", st);
    if (accum)
      hipLaunchKernelGGL((k_conv_fwd<V, CPL, true>), dim3(grid), dim3(kWave), 0, st, a);
    else
      hipLaunchKernelGGL((k_conv_fwd<V, CPL, false>), dim3(grid), dim3(kWave), 0, st, a);
  }
  E3_HIP(hipGetLastError());
  return E3_OK;
}

// The double backward's three forward terms in one launch (k_conv_fwd3):
// m = conv(x2, y, s) + conv(x, y2, s) + conv(x, y, s2), overwritten.
template <class V>
e3_status run_fwd3(const e3_plan* p, const e3_graph* g, const float* x, const float* x2, const float* y,
                   const float* y2, const float* s, const float* s2, float* m, hipStream_t st) {
  ConvArgs a = base_args(p, g);
  a.x = x, a.x2 = x2, a.y = y, a.y2 = y2, a.s = s, a.s2 = s2, a.m = m;
  a.nslab = (a.C + kWave - 1) / kWave;  // one channel per lane
  if (g->n_nodes == 0) return E3_OK;
  const unsigned grid = (unsigned)(kXcd * a.chunk * V::NFG * a.nslab);
  {
    TimedLaunch t_("conv_fwd3", st);
    hipLaunchKernelGGL((k_conv_fwd3<V>), dim3(grid), dim3(kWave), 0, st, a);
  }
  E3_HIP(hipGetLastError());
  return E3_OK;
}

// One backward convolution.  Harmonics from y when given (then dy is the
// harmonic cotangent output), else from vec (then dvec = J^T dy).  Any of
// dx, dvec/dy, ds may be null: that cotangent is not stored.  accum is a mask
// of kAccDx / kAccDy / kAccDs: those cotangents are added to the outputs'
// contents instead of overwriting them.
constexpr int kAccDx = 1, kAccDy = 2, kAccDs = 4;

template <class V, int CPLX>
e3_status run_bwd(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* y,
                  const float* s, const float* dm, float* dx, float* dvec, float* dy, float* ds, int accum, void* ws,
                  hipStream_t st) {
  if (g->n_nodes == 0) return E3_OK;
  Ws w = bwd_ws<V>(p, g);
  ConvArgs a = base_args(p, g);
  a.x = x, a.vec = vec, a.y = y, a.s = s, a.dm = dm, a.accum = (accum & kAccDs) != 0;
  a.T = reinterpret_cast<float*>(ws);
  a.DY = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + w.t_bytes);  // always written
  a.ds = ds ? ds : a.DY;
  a.ds_row = ds ? (int64_t)V::NP * a.C * 4 : 0;
  a.t_row = dx ? (int64_t)V::D_IN * a.C * 4 : 0;
  a.nslab = p->nslab_b;
  if (g->n_live > 0) {
    const unsigned grid = (unsigned)(kXcd * a.chunk * V::NBG * a.nslab);
    TimedLaunch t_("conv_bwd_edges", st);
    if (p->cpl_b == 1) {
      if (a.accum)
        hipLaunchKernelGGL((k_conv_bwd_edges<V, 1, true>), dim3(grid), dim3(kWave), 0, st, a);
      else
        hipLaunchKernelGGL((k_conv_bwd_edges<V, 1, false>), dim3(grid), dim3(kWave), 0, st, a);
    } else {
      if (a.accum)
        hipLaunchKernelGGL((k_conv_bwd_edges<V, E3_BWD_CPL, true>), dim3(grid), dim3(kWave), 0, st, a);
      else
        hipLaunchKernelGGL((k_conv_bwd_edges<V, E3_BWD_CPL, false>), dim3(grid), dim3(kWave), 0, st, a);
    }
    E3_HIP(hipGetLastError());
  }
  if (dx) {
    TimedLaunch t_("conv_bwd_dx", st);
    const int flat4 = V::D_IN * a.C / 4;
    const int nsl = (flat4 + kWave * kDxVec - 1) / (kWave * kDxVec);
    hipLaunchKernelGGL(k_conv_bwd_dx, dim3((unsigned)(kXcd * a.chunk * nsl)), dim3(kWave), 0, st, a.T, dx,
                       g->rowptr_s, a.n_nodes, a.chunk, flat4, nsl, (accum & kAccDx) != 0);
    E3_HIP(hipGetLastError());
  }
  if (g->n_live > 0 && dvec) {
    TimedLaunch t_("conv_bwd_dvec", st);
    hipLaunchKernelGGL((k_conv_bwd_dvec<V>), dim3(blocks_for(g->n_live, 256)), dim3(256), 0, st, vec, a.DY, g->eid_r,
                       dvec, g->n_live, p->nslab_b);
    E3_HIP(hipGetLastError());
  }
  if (g->n_live > 0 && dy) {
    TimedLaunch t_("conv_bwd_dy", st);
    hipLaunchKernelGGL((k_conv_bwd_dy<V>), dim3(blocks_for(g->n_live * V::D_SH, 256)), dim3(256), 0, st, a.DY,
                       g->eid_r, dy, g->n_live, p->nslab_b, (accum & kAccDy) != 0);
    E3_HIP(hipGetLastError());
  }
  // padding edges: zero cotangents (left unchanged when accumulating)
  float* z0 = (accum & kAccDs) ? nullptr : ds;
  float* z1 = dvec ? dvec : ((accum & kAccDy) ? nullptr : dy);
  const int64_t w1 = dvec ? 3 : V::D_SH;
  if (g->n_pad > 0 && (z0 || z1)) {
    TimedLaunch t_("conv_bwd_pad", st);
    hipLaunchKernelGGL(k_zero_pad, dim3((unsigned)g->n_pad), dim3(256), 0, st, g->eid_r + g->n_live, g->n_pad, z0,
                       (int64_t)V::NP * a.C, z1, w1);
    E3_HIP(hipGetLastError());
  }
  return E3_OK;
}

// The double backward's three backward terms in one sweep (k_conv_bwd3),
// then the sender segment sum (gx) and the harmonic cotangent sum (gy); all
// three outputs overwritten.  One channel per lane: the workspace layout of
// e3_conv_bwd with one channel per lane (cpl_b == 1).
template <class V>
e3_status run_bwd3(const e3_plan* p, const e3_graph* g, const float* x, const float* x2, const float* y,
                   const float* y2, const float* s, const float* s2, const float* dm, float* gx, float* gy,
                   float* gs, void* ws, hipStream_t st) {
  if (g->n_nodes == 0) return E3_OK;
  if (p->cpl_b != 1) return E3_ERR_UNSUPPORTED;
  Ws w = bwd_ws<V>(p, g);
  ConvArgs a = base_args(p, g);
  a.x = x, a.x2 = x2, a.y = y, a.y2 = y2, a.s = s, a.s2 = s2, a.dm = dm, a.ds = gs;
  a.T = reinterpret_cast<float*>(ws);
  a.DY = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + w.t_bytes);
  a.nslab = p->nslab_b;
  if (g->n_live > 0) {
    const unsigned grid = (unsigned)(kXcd * a.chunk * V::NBG * a.nslab);
    TimedLaunch t_("conv_bwd3", st);
    hipLaunchKernelGGL((k_conv_bwd3<V>), dim3(grid), dim3(kWave), 0, st, a);
    E3_HIP(hipGetLastError());
  }
  {
    TimedLaunch t_("conv_bwd_dx", st);
    const int flat4 = V::D_IN * a.C / 4;
    const int nsl = (flat4 + kWave * kDxVec - 1) / (kWave * kDxVec);
    hipLaunchKernelGGL(k_conv_bwd_dx, dim3((unsigned)(kXcd * a.chunk * nsl)), dim3(kWave), 0, st, a.T, gx,
                       g->rowptr_s, a.n_nodes, a.chunk, flat4, nsl, 0);
    E3_HIP(hipGetLastError());
  }
  if (g->n_live > 0) {
    TimedLaunch t_("conv_bwd_dy", st);
    hipLaunchKernelGGL((k_conv_bwd_dy<V>), dim3(blocks_for(g->n_live * V::D_SH, 256)), dim3(256), 0, st, a.DY,
                       g->eid_r, gy, g->n_live, p->nslab_b, 0);
    E3_HIP(hipGetLastError());
  }
  if (g->n_pad > 0) {  // padding edges: zero cotangents
    TimedLaunch t_("conv_bwd_pad", st);
    hipLaunchKernelGGL(k_zero_pad, dim3((unsigned)g->n_pad), dim3(256), 0, st, g->eid_r + g->n_live, g->n_pad, gs,
                       (int64_t)V::NP * a.C, gy, (int64_t)V::D_SH);
    E3_HIP(hipGetLastError());
  }
  return E3_OK;
}

template <class V, int CPL>
e3_status run_tp(const e3_plan* p, const float* x, const float* y, const float* w, float* z, int64_t rows,
                 hipStream_t st) {
  if (rows == 0) return E3_OK;
  {
    TimedLaunch t_("tp_fwd", st);
    const dim3 grid((unsigned)tile_grid(false, rows, kTpRows, p->nslab_f));
    hipLaunchKernelGGL((k_tp<V, CPL>), grid, dim3(kWave), 0, st, x, y, w, z, rows, p->lay.C, p->nslab_f);
  }
  E3_HIP(hipGetLastError());
  return E3_OK;
}

template <class V, int CPL>
e3_status run_tp_bwd(const e3_plan* p, const float* x, const float* y, const float* w, const float* dz, float* dx,
                     float* dy, float* dw, void* ws, int64_t rows, hipStream_t st) {
  if (rows == 0) return E3_OK;
  TpbArgs a{};
  a.x = x, a.y = y, a.w = w, a.dz = dz, a.dx = dx, a.dw = dw;
  a.DY = reinterpret_cast<float*>(ws);
  a.rows = rows;
  a.C = p->lay.C;
  a.nslab = p->nslab_b;
  {
    TimedLaunch t_("tp_bwd", st);
    // the (group, slab) waves of a row tile on one XCD: 3.42 -> 3.33 ms at 200,000 rows, l <= 3
    const dim3 grid((unsigned)tile_grid(E3_TP_XCD, rows, kTpRows, V::NBG * a.nslab));
    hipLaunchKernelGGL((k_tp_bwd<V, CPL>), grid, dim3(kWave), 0, st, a);
  }
  E3_HIP(hipGetLastError());
  {
    TimedLaunch t_("tp_bwd_dy", st);
    hipLaunchKernelGGL((k_tp_bwd_dy<V>), dim3(blocks_for(rows, 256)), dim3(256), 0, st, a.DY, dy, rows, a.nslab);
  }
  E3_HIP(hipGetLastError());
  return E3_OK;
}

// Scratch of the radial backward: T and DY as in the plain backward, then ds
// by edge id (all E rows when any edge is live), the dW partials of each row
// chunk and the dh partials of each column slab.
struct RadWs {
  size_t t, dy, ds, dwp, dhp;
  int nchunk, rows_per, nsl4, nv, pc4;
  size_t total() const { return t + dy + ds + dwp + dhp; }
};

template <class V>
RadWs rad_ws(const e3_plan* p, const e3_graph* g, int K) {
  RadWs w{};
  const Ws b = bwd_ws<V>(p, g);
  w.t = b.t_bytes, w.dy = b.dy_bytes;
  const int64_t pc = (int64_t)V::NP * p->lay.C, nl = g->n_live > 0 ? g->n_edges : 0;
  w.pc4 = (int)(pc / 4);
  w.nsl4 = (w.pc4 + kWave * kGradF - 1) / (kWave * kGradF);
  w.nv = K <= 8 ? 8 : 16;
  // about 8k waves in the gradient kernel, at least 256 rows each
  const int64_t want = std::max<int64_t>(1, 8192 / w.nsl4);
  const int64_t nch = std::min<int64_t>(want, std::max<int64_t>(1, (nl + 255) / 256));
  w.rows_per = (int)std::max<int64_t>(1, (nl + nch - 1) / nch);
  w.nchunk = (int)((nl + w.rows_per - 1) / w.rows_per);
  w.ds = align256((size_t)nl * pc * sizeof(float));
  w.dwp = align256((size_t)w.nchunk * K * pc * sizeof(float));
  w.dhp = align256((size_t)nl * w.nsl4 * w.nv * sizeof(float));
  return w;
}

template <class V>
e3_status run_fwd_rad(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* h,
                      const float* W, int K, float* m, hipStream_t st) {
  if (g->n_nodes == 0) return E3_OK;
  ConvArgs a = base_args(p, g);
  a.x = x, a.vec = vec, a.h = h, a.W = W, a.K = K, a.m = m;
  a.nslab = p->nslab_b;
  const unsigned grid = (unsigned)(kXcd * a.chunk * V::NFG * a.nslab);
  {
    TimedLaunch t_("conv_fwd_rad", st);
    if (K <= 8 && E3_RAD_WREG)
      hipLaunchKernelGGL((k_conv_fwd_rad<V, 8>), dim3(grid), dim3(kWave), 0, st, a);
    else
      hipLaunchKernelGGL((k_conv_fwd_rad<V, 0>), dim3(grid), dim3(kWave), 0, st, a);
  }
  E3_HIP(hipGetLastError());
  return E3_OK;
}

template <class V>
e3_status run_bwd_rad(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* h,
                      const float* W, int K, const float* dm, float* dx, float* dvec, float* dh, float* dW, void* ws,
                      hipStream_t st) {
  const RadWs w = rad_ws<V>(p, g, K);
  char* base = reinterpret_cast<char*>(ws);
  ConvArgs a = base_args(p, g);
  a.x = x, a.vec = vec, a.h = h, a.W = W, a.K = K, a.dm = dm;
  a.T = reinterpret_cast<float*>(base);
  a.DY = reinterpret_cast<float*>(base + w.t);
  a.ds = reinterpret_cast<float*>(base + w.t + w.dy);
  float* dWp = reinterpret_cast<float*>(base + w.t + w.dy + w.ds);
  float* DHp = reinterpret_cast<float*>(base + w.t + w.dy + w.ds + w.dwp);
  a.nslab = p->nslab_b;
  if (g->n_live > 0) {
    const unsigned grid = (unsigned)(kXcd * a.chunk * V::NBG * a.nslab);
    TimedLaunch t_("conv_bwd_rad_edges", st);
    hipLaunchKernelGGL((k_conv_bwd_rad<V>), dim3(grid), dim3(kWave), 0, st, a);
    E3_HIP(hipGetLastError());
  }
  if (g->n_nodes > 0) {
    TimedLaunch t_("conv_bwd_dx", st);
    const int flat4 = V::D_IN * a.C / 4;
    const int nsl = (flat4 + kWave * kDxVec - 1) / (kWave * kDxVec);
    hipLaunchKernelGGL(k_conv_bwd_dx, dim3((unsigned)(kXcd * a.chunk * nsl)), dim3(kWave), 0, st, a.T, dx,
                       g->rowptr_s, a.n_nodes, a.chunk, flat4, nsl, 0);
    E3_HIP(hipGetLastError());
  }
  if (g->n_live > 0) {
    {
      TimedLaunch t_("conv_bwd_dvec", st);
      hipLaunchKernelGGL((k_conv_bwd_dvec<V>), dim3(blocks_for(g->n_live, 256)), dim3(256), 0, st, vec, a.DY,
                         g->eid_r, dvec, g->n_live, p->nslab_b);
      E3_HIP(hipGetLastError());
    }
    if (g->n_pad > 0) {
      // the ds rows of padding edges enter the gradient sums: clear them
      TimedLaunch t_("rad_pad_ds", st);
      hipLaunchKernelGGL(k_zero_pad, dim3((unsigned)g->n_pad), dim3(256), 0, st, g->eid_r + g->n_live, g->n_pad,
                         a.ds, (int64_t)w.pc4 * 4, dvec, (int64_t)3);
      E3_HIP(hipGetLastError());
    }
    const int64_t E = g->n_edges;
    {
      TimedLaunch t_("rad_grad", st);
      const dim3 grid((unsigned)((int64_t)w.nchunk * w.nsl4));
      if (K <= 8)
        hipLaunchKernelGGL(k_rad_grad<2>, grid, dim3(kWave), 0, st, a.ds, h, W, dWp, DHp, E, w.pc4, K, w.nsl4,
                           w.rows_per);
      else
        hipLaunchKernelGGL(k_rad_grad<4>, grid, dim3(kWave), 0, st, a.ds, h, W, dWp, DHp, E, w.pc4, K, w.nsl4,
                           w.rows_per);
      E3_HIP(hipGetLastError());
    }
    {
      TimedLaunch t_("rad_dh_sum", st);
      hipLaunchKernelGGL(k_rad_dh_sum, dim3(blocks_for(E * w.nv, 256)), dim3(256), 0, st, DHp, dh, E, K, w.nsl4,
                         w.nv);
      E3_HIP(hipGetLastError());
    }
  }
  {
    const int64_t n = (int64_t)K * w.pc4 * 4;
    TimedLaunch t_("rad_dw_sum", st);
    hipLaunchKernelGGL(k_rad_dw_sum, dim3(blocks_for(n, 256)), dim3(256), 0, st, dWp, dW, n, w.nchunk);
    E3_HIP(hipGetLastError());
  }
  if (g->n_pad > 0) {
    TimedLaunch t_("conv_bwd_pad", st);
    hipLaunchKernelGGL(k_zero_pad, dim3((unsigned)g->n_pad), dim3(256), 0, st, g->eid_r + g->n_live, g->n_pad, dh,
                       (int64_t)K, dvec, (int64_t)3);
    E3_HIP(hipGetLastError());
  }
  return E3_OK;
}

template <class V>
size_t tp_ws(const e3_plan* p, int64_t rows) {
  return align256((size_t)rows * V::NBG * p->nslab_b * 16 * sizeof(float));
}

struct VariantOps {
  const char* sig;
  int d_in, d_sh, d_out, np, lsh, nbg;
  e3_status (*fwd[2])(const e3_plan*, const e3_graph*, const float*, const float*, const float*, const float*,
                      float*, int, hipStream_t);
  e3_status (*bwd[2])(const e3_plan*, const e3_graph*, const float*, const float*, const float*, const float*,
                      const float*, float*, float*, float*, float*, int, void*, hipStream_t);
  e3_status (*tp[2])(const e3_plan*, const float*, const float*, const float*, float*, int64_t, hipStream_t);
  Ws (*ws)(const e3_plan*, const e3_graph*);
  e3_status (*tpb)(const e3_plan*, const float*, const float*, const float*, const float*, float*, float*, float*,
                   void*, int64_t, hipStream_t);
  size_t (*tpws)(const e3_plan*, int64_t);
  e3_status (*rfwd)(const e3_plan*, const e3_graph*, const float*, const float*, const float*, const float*, int,
                    float*, hipStream_t);
  e3_status (*rbwd)(const e3_plan*, const e3_graph*, const float*, const float*, const float*, const float*, int,
                    const float*, float*, float*, float*, float*, void*, hipStream_t);
  RadWs (*rws)(const e3_plan*, const e3_graph*, int);
  e3_status (*fwd3)(const e3_plan*, const e3_graph*, const float*, const float*, const float*, const float*,
                    const float*, const float*, float*, hipStream_t);
  e3_status (*bwd3)(const e3_plan*, const e3_graph*, const float*, const float*, const float*, const float*,
                    const float*, const float*, const float*, float*, float*, float*, void*, hipStream_t);
};

#define E3_VARIANT(V)                                                                                    \
  VariantOps{e3gen::V::SIG,                                                                              \
             e3gen::V::D_IN,                                                                             \
             e3gen::V::D_SH,                                                                             \
             e3gen::V::D_OUT,                                                                            \
             e3gen::V::NP,                                                                               \
             e3gen::V::LSH,                                                                              \
             e3gen::V::NBG,                                                                              \
             {&run_fwd<e3gen::V, 1>, &run_fwd<e3gen::V, 2>},                                             \
             {&run_bwd<e3gen::V, 1>, &run_bwd<e3gen::V, 2>},                                             \
             {&run_tp<e3gen::V, 1>, &run_tp<e3gen::V, 2>},                                               \
             &bwd_ws<e3gen::V>,                                                                          \
             &run_tp_bwd<e3gen::V, 1>,                                                                   \
             &tp_ws<e3gen::V>,                                                                           \
             &run_fwd_rad<e3gen::V>,                                                                     \
             &run_bwd_rad<e3gen::V>,                                                                     \
             &rad_ws<e3gen::V>,                                                                          \
             &run_fwd3<e3gen::V>,                                                                        \
             &run_bwd3<e3gen::V>},

const VariantOps kVariants[] = {E3GEN_FOR_EACH_VARIANT(E3_VARIANT)};
constexpr int kNumVariants = sizeof(kVariants) / sizeof(kVariants[0]);

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int cpl_index(int cpl) { return cpl == 1 ? 0 : 1; }
int cpl_of(const e3_plan* p) { return p->cpl_f; }

e3_status check_plan(const e3_plan* p) {
  if (!p) return E3_ERR_INVALID_ARG;
  if (p->variant < 0) return E3_ERR_UNSUPPORTED;
  return E3_OK;
}

}  // namespace

// ============================================================ C ABI
extern "C" {

const char* e3_status_str(e3_status s) {
  switch (s) {
    case E3_OK: return "ok";
    case E3_ERR_INVALID_ARG: return "invalid argument";
    case E3_ERR_UNSUPPORTED: return "unsupported configuration";
    case E3_ERR_INDEX_OUT_OF_RANGE: return "edge index out of range";
    case E3_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case E3_ERR_HIP: return "HIP runtime error";
    case E3_ERR_ALLOC: return "allocation failed";
  }
  return "unknown status";
}

const char* e3_last_error(void) { return g_last_error.c_str(); }

e3_status e3_timing_enable(int on) {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  g_timing.on = on != 0;
  return E3_OK;
}

e3_status e3_timing_reset(void) {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  for (auto& p : g_timing.pending) {
    (void)hipEventSynchronize(p.b);
    g_timing.pool.push_back(p.a);
    g_timing.pool.push_back(p.b);
  }
  g_timing.pending.clear();
  g_timing.acc.clear();
  return E3_OK;
}

e3_status e3_timing_read(int cap, char* names, double* ms, int64_t* count, int* n) {
  if (cap < 0 || !n || (cap > 0 && (!names || !ms || !count))) return E3_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(g_timing.mu);
  for (auto& p : g_timing.pending) {
    E3_HIP(hipEventSynchronize(p.b));
    float t = 0.0f;
    E3_HIP(hipEventElapsedTime(&t, p.a, p.b));
    auto& slot = g_timing.acc[p.name];
    slot.first += t;
    slot.second += 1;
    g_timing.pool.push_back(p.a);
    g_timing.pool.push_back(p.b);
  }
  g_timing.pending.clear();
  int i = 0;
  for (const auto& [name, v] : g_timing.acc) {
    if (i < cap) {
      std::memset(names + 32 * i, 0, 32);
      std::strncpy(names + 32 * i, name.c_str(), 31);
      ms[i] = v.first;
      count[i] = v.second;
    }
    ++i;
  }
  *n = i;
  return E3_OK;
}

e3_status e3_plan_create(const char* irreps_x, int lmax_sh, int lmax_out, unsigned flags, e3_plan** out) {
  if (!irreps_x || !out) return E3_ERR_INVALID_ARG;
  *out = nullptr;
  if (lmax_sh < 0 || lmax_sh > 3 || lmax_out < 0 || lmax_out > 16 || flags > 1u) return E3_ERR_INVALID_ARG;
  std::vector<e3b::Block> blocks;
  std::string err;
  if (!e3b::parse_irreps(irreps_x, blocks, err)) {
    g_last_error = err;
    return E3_ERR_INVALID_ARG;
  }
  for (const auto& b : blocks)
    if (b.l > 16) return E3_ERR_INVALID_ARG;
  e3_plan* p = new (std::nothrow) e3_plan();
  if (!p) return E3_ERR_ALLOC;
  if (!e3b::make_layout(irreps_x, lmax_sh, lmax_out, flags == E3_PARITY_NATURAL, p->lay, err)) {
    g_last_error = err;
    delete p;
    return E3_ERR_UNSUPPORTED;
  }
  try {
    p->recs = e3b::coo(p->lay);
  } catch (const std::exception& ex) {
    g_last_error = ex.what();
    delete p;
    return E3_ERR_UNSUPPORTED;
  }
  const std::string sig = e3b::path_signature(p->lay);
  // Channels: multiples of 4 up to kMaxChannels.  The forward, tensor-product
  // and dx kernels give each lane 2 consecutive channels when C > 64 (one lane
  // per channel otherwise); the backward sweep gives each lane 1.  Channels
  // beyond one wave are covered by further 64-lane slabs.
  const int C = p->lay.C;
  if (C >= 4 && C % 4 == 0 && C <= kMaxChannels) {
    for (int i = 0; i < kNumVariants; ++i)
      if (sig == kVariants[i].sig && p->lay.d_sh == kVariants[i].d_sh) p->variant = i;
  }
  if (p->variant >= 0) {
    p->cpl_f = C <= kWave ? 1 : E3_FWD_CPL;
    p->nslab_f = (C + kWave * p->cpl_f - 1) / (kWave * p->cpl_f);
    p->cpl_b = C <= kWave ? 1 : E3_BWD_CPL;
    p->nslab_b = (C + kWave * p->cpl_b - 1) / (kWave * p->cpl_b);
  }
  *out = p;
  return E3_OK;
}

e3_status e3_plan_query(const e3_plan* p, e3_plan_info* info) {
  if (!p || !info) return E3_ERR_INVALID_ARG;
  info->C = p->lay.C;
  info->P = (int)p->lay.paths.size();
  info->D_in = p->lay.d_in;
  info->D_sh = p->lay.d_sh;
  info->D_out = p->lay.d_out;
  info->nnz = (int)p->recs.size();
  info->lmax_sh = p->lay.lmax_sh;
  info->lmax_out = p->lay.lmax_out;
  info->supported = p->variant >= 0 ? 1 : 0;
  return E3_OK;
}

e3_status e3_plan_destroy(e3_plan* p) {
  delete p;
  return E3_OK;
}

e3_status e3_plan_paths(const e3_plan* p, int32_t* out) {
  if (!p || !out) return E3_ERR_INVALID_ARG;
  for (size_t i = 0; i < p->lay.paths.size(); ++i) {
    const auto& q = p->lay.paths[i];
    const int32_t v[7] = {q.l1, q.l2, q.l3, q.p3, q.x_off, q.y_off, q.out_off};
    std::memcpy(out + 7 * i, v, sizeof(v));
  }
  return E3_OK;
}

e3_status e3_plan_records(const e3_plan* p, int64_t cap, int32_t* i0, int32_t* i1, int32_t* i2, double* val,
                          int64_t* n) {
  if (!p || !n || cap < 0) return E3_ERR_INVALID_ARG;
  *n = (int64_t)p->recs.size();
  const int64_t m = std::min<int64_t>(cap, *n);
  if (m > 0 && (!i0 || !i1 || !i2 || !val)) return E3_ERR_INVALID_ARG;
  for (int64_t k = 0; k < m; ++k) {
    i0[k] = p->recs[k].i0, i1[k] = p->recs[k].i1, i2[k] = p->recs[k].i2, val[k] = p->recs[k].v;
  }
  return E3_OK;
}

e3_status e3_sh_host(int lmax, const double* u, double* y, int64_t n) {
  if (lmax < 0 || lmax > 3 || n < 0 || (n > 0 && (!u || !y))) return E3_ERR_INVALID_ARG;
  e3b::ShTable t = e3b::sh_table(lmax);
  const int d = (lmax + 1) * (lmax + 1);
  for (int64_t i = 0; i < n; ++i) e3b::sh_eval(t, u + 3 * i, y + d * i);
  return E3_OK;
}

e3_status e3_graph_create(const int32_t* sender, const int32_t* receiver, int64_t n_nodes, int64_t n_edges,
                          int32_t pad_node, e3_stream stream, e3_graph** out) {
  if (!out) return E3_ERR_INVALID_ARG;
  *out = nullptr;
  if (n_nodes < 0 || n_edges < 0 || n_nodes >= INT32_MAX || n_edges >= INT32_MAX) return E3_ERR_INVALID_ARG;
  if (n_edges > 0 && (!sender || !receiver)) return E3_ERR_INVALID_ARG;
  if (pad_node < -1 || (pad_node >= 0 && pad_node >= n_nodes)) return E3_ERR_INVALID_ARG;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  e3_graph* g = new (std::nothrow) e3_graph();
  if (!g) return E3_ERR_ALLOC;
  g->n_nodes = n_nodes, g->n_edges = n_edges, g->pad = pad_node;
  const int64_t E = n_edges, N = n_nodes;
  auto fail = [&](e3_status s) {
    e3_graph_destroy(g);
    return s;
  };
  auto alloc = [&](void** p, size_t bytes) -> bool {
    if (hipMalloc(p, std::max<size_t>(bytes, 4)) != hipSuccess) {
      g_last_error = "hipMalloc failed in e3_graph_create";
      return false;
    }
    return true;
  };
  if (!alloc((void**)&g->rowptr_r, (N + 1) * 4) || !alloc((void**)&g->rowptr_s, (N + 1) * 4) ||
      !alloc((void**)&g->eid_r, E * 4) || !alloc((void**)&g->eid_s, E * 4) || !alloc((void**)&g->src_r, E * 4) ||
      !alloc((void**)&g->r2s, E * 4) || !alloc((void**)&g->pos_s, E * 4))
    return fail(E3_ERR_ALLOC);
  uint32_t *key_r = nullptr, *key_s = nullptr, *key_sorted = nullptr;
  int32_t* ids = nullptr;
  int* flag = nullptr;
  void* tmp = nullptr;
  auto cleanup = [&]() {
    (void)hipFree(key_r), (void)hipFree(key_s), (void)hipFree(key_sorted), (void)hipFree(ids), (void)hipFree(flag),
        (void)hipFree(tmp);
  };
  if (!alloc((void**)&key_r, E * 4) || !alloc((void**)&key_s, E * 4) || !alloc((void**)&key_sorted, E * 4) ||
      !alloc((void**)&ids, E * 4) || !alloc((void**)&flag, 2 * sizeof(int))) {
    cleanup();
    return fail(E3_ERR_ALLOC);
  }
  int end_bit = 1;
  while (end_bit < 32 && ((int64_t)1 << end_bit) <= N) ++end_bit;
  size_t tmp_bytes = 0;
  hipError_t herr = hipSuccess;
  herr = hipMemsetAsync(flag, 0, 2 * sizeof(int), st);
  if (herr == hipSuccess && E > 0) {
    hipLaunchKernelGGL(k_graph_keys, dim3(blocks_for(E, 256)), dim3(256), 0, st, sender, receiver, E, (int32_t)N,
                       pad_node, key_r, key_s, ids, flag);
    herr = hipGetLastError();
    if (herr == hipSuccess)
      herr = hipcub::DeviceRadixSort::SortPairs(nullptr, tmp_bytes, key_r, key_sorted, ids, g->eid_r, (int)E, 0,
                                                end_bit, st);
    if (herr == hipSuccess && !alloc(&tmp, tmp_bytes)) {
      cleanup();
      return fail(E3_ERR_ALLOC);
    }
    if (herr == hipSuccess)
      herr = hipcub::DeviceRadixSort::SortPairs(tmp, tmp_bytes, key_r, key_sorted, ids, g->eid_r, (int)E, 0, end_bit,
                                                st);
    if (herr == hipSuccess) {
      hipLaunchKernelGGL(k_graph_rowptr, dim3(blocks_for(N + 1, 256)), dim3(256), 0, st, key_sorted, E, (int32_t)N,
                         g->rowptr_r);
      herr = hipGetLastError();
    }
    if (herr == hipSuccess)
      herr = hipcub::DeviceRadixSort::SortPairs(tmp, tmp_bytes, key_s, key_sorted, ids, g->eid_s, (int)E, 0, end_bit,
                                                st);
    if (herr == hipSuccess) {
      hipLaunchKernelGGL(k_graph_rowptr, dim3(blocks_for(N + 1, 256)), dim3(256), 0, st, key_sorted, E, (int32_t)N,
                         g->rowptr_s);
      herr = hipGetLastError();
    }
  } else if (herr == hipSuccess) {
    herr = hipMemsetAsync(g->rowptr_r, 0, (N + 1) * 4, st);
    if (herr == hipSuccess) herr = hipMemsetAsync(g->rowptr_s, 0, (N + 1) * 4, st);
  }
  int host[2] = {0, 0};
  if (herr == hipSuccess) herr = hipMemcpyAsync(&host[0], flag, sizeof(int), hipMemcpyDeviceToHost, st);
  if (herr == hipSuccess) herr = hipMemcpyAsync(&host[1], g->rowptr_r + N, sizeof(int), hipMemcpyDeviceToHost, st);
  if (herr == hipSuccess) herr = hipStreamSynchronize(st);
  if (herr != hipSuccess) {
    g_last_error = std::string("e3_graph_create: ") + hipGetErrorString(herr);
    cleanup();
    return fail(E3_ERR_HIP);
  }
  if (host[0]) {
    cleanup();
    return fail(E3_ERR_INDEX_OUT_OF_RANGE);
  }
  g->n_live = host[1];
  g->n_pad = E - g->n_live;
  if (g->n_live > 0) {
    hipLaunchKernelGGL(k_graph_finish, dim3(blocks_for(g->n_live, 256)), dim3(256), 0, st, sender, g->eid_r, g->eid_s,
                       g->n_live, g->src_r, g->pos_s);
    herr = hipGetLastError();
    if (herr == hipSuccess) {
      hipLaunchKernelGGL(k_graph_r2s, dim3(blocks_for(g->n_live, 256)), dim3(256), 0, st, g->eid_r, g->pos_s,
                         g->n_live, g->r2s);
      herr = hipGetLastError();
    }
    if (herr == hipSuccess) herr = hipStreamSynchronize(st);  // temporaries are freed below
  }
  cleanup();
  if (herr != hipSuccess) {
    g_last_error = std::string("e3_graph_create: ") + hipGetErrorString(herr);
    return fail(E3_ERR_HIP);
  }
  *out = g;
  return E3_OK;
}

e3_status e3_graph_live_edges(const e3_graph* g, int64_t* n_live) {
  if (!g || !n_live) return E3_ERR_INVALID_ARG;
  *n_live = g->n_live;
  return E3_OK;
}

e3_status e3_graph_export(const e3_graph* g, int32_t* perm_r, int32_t* rowptr_r, int32_t* perm_s, int32_t* rowptr_s) {
  if (!g) return E3_ERR_INVALID_ARG;
  const size_t nl = (size_t)g->n_live * 4, nr = (size_t)(g->n_nodes + 1) * 4;
  if (perm_r && nl) E3_HIP(hipMemcpy(perm_r, g->eid_r, nl, hipMemcpyDeviceToDevice));
  if (rowptr_r) E3_HIP(hipMemcpy(rowptr_r, g->rowptr_r, nr, hipMemcpyDeviceToDevice));
  if (perm_s && nl) E3_HIP(hipMemcpy(perm_s, g->eid_s, nl, hipMemcpyDeviceToDevice));
  if (rowptr_s) E3_HIP(hipMemcpy(rowptr_s, g->rowptr_s, nr, hipMemcpyDeviceToDevice));
  return E3_OK;
}

e3_status e3_graph_destroy(e3_graph* g) {
  if (!g) return E3_OK;
  (void)hipFree(g->rowptr_r), (void)hipFree(g->eid_r), (void)hipFree(g->src_r), (void)hipFree(g->r2s);
  (void)hipFree(g->rowptr_s), (void)hipFree(g->eid_s), (void)hipFree(g->pos_s);
  delete g;
  return E3_OK;
}

e3_status e3_sh(int lmax, const float* vec, float* y, int64_t n, e3_stream stream) {
  if (lmax < 0 || lmax > 3 || n < 0 || (n > 0 && (!vec || !y))) return E3_ERR_INVALID_ARG;
  if (n == 0) return E3_OK;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const dim3 grid(blocks_for(n, 256));
  TimedLaunch t_("sh", st);
  switch (lmax) {
    case 0: hipLaunchKernelGGL(k_sh<0>, grid, dim3(256), 0, st, vec, y, n); break;
    case 1: hipLaunchKernelGGL(k_sh<1>, grid, dim3(256), 0, st, vec, y, n); break;
    case 2: hipLaunchKernelGGL(k_sh<2>, grid, dim3(256), 0, st, vec, y, n); break;
    default: hipLaunchKernelGGL(k_sh<3>, grid, dim3(256), 0, st, vec, y, n); break;
  }
  E3_HIP(hipGetLastError());
  return E3_OK;
}

e3_status e3_sh_bwd(int lmax, const float* vec, const float* dy, float* dvec, int64_t n, e3_stream stream) {
  if (lmax < 0 || lmax > 3 || n < 0 || (n > 0 && (!vec || !dy || !dvec))) return E3_ERR_INVALID_ARG;
  if (n == 0) return E3_OK;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const dim3 grid(blocks_for(n, 256));
  TimedLaunch t_("sh_bwd", st);
  switch (lmax) {
    case 0: hipLaunchKernelGGL(k_sh_bwd<0>, grid, dim3(256), 0, st, vec, dy, dvec, n); break;
    case 1: hipLaunchKernelGGL(k_sh_bwd<1>, grid, dim3(256), 0, st, vec, dy, dvec, n); break;
    case 2: hipLaunchKernelGGL(k_sh_bwd<2>, grid, dim3(256), 0, st, vec, dy, dvec, n); break;
    default: hipLaunchKernelGGL(k_sh_bwd<3>, grid, dim3(256), 0, st, vec, dy, dvec, n); break;
  }
  E3_HIP(hipGetLastError());
  return E3_OK;
}

e3_status e3_tp_fwd(const e3_plan* p, const float* x, const float* y, const float* w, float* z, int64_t rows,
                    e3_stream stream) {
  e3_status s = check_plan(p);
  if (s != E3_OK) return s;
  if (rows < 0) return E3_ERR_INVALID_ARG;
  if (rows > 0 && (!x || !y || !w || !z || !aligned16(x) || !aligned16(w) || !aligned16(z))) return E3_ERR_INVALID_ARG;
  if (rows == 0) return E3_OK;
  const VariantOps& v = kVariants[p->variant];
  return v.tp[cpl_index(cpl_of(p))](p, x, y, w, z, rows, reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_tp_workspace_size(const e3_plan* p, int64_t rows, size_t* bwd_bytes) {
  e3_status s = check_plan(p);
  if (s != E3_OK) return s;
  if (rows < 0 || !bwd_bytes) return E3_ERR_INVALID_ARG;
  *bwd_bytes = kVariants[p->variant].tpws(p, rows);
  return E3_OK;
}

e3_status e3_tp_bwd(const e3_plan* p, const float* x, const float* y, const float* w, const float* dz, float* dx,
                    float* dy, float* dw, void* ws, size_t ws_bytes, int64_t rows, e3_stream stream) {
  e3_status s = check_plan(p);
  if (s != E3_OK) return s;
  if (rows < 0) return E3_ERR_INVALID_ARG;
  if (rows == 0) return E3_OK;
  if (!x || !y || !w || !dz || !dx || !dy || !dw || !ws || !aligned16(x) || !aligned16(w) || !aligned16(dz) ||
      !aligned16(dx) || !aligned16(dw) || !aligned16(ws))
    return E3_ERR_INVALID_ARG;
  const VariantOps& v = kVariants[p->variant];
  if (ws_bytes < v.tpws(p, rows)) return E3_ERR_WORKSPACE_TOO_SMALL;
  return v.tpb(p, x, y, w, dz, dx, dy, dw, ws, rows, reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_conv_workspace_size(const e3_plan* p, const e3_graph* g, size_t* fwd_bytes, size_t* bwd_bytes) {
  e3_status s = check_plan(p);
  if (s != E3_OK) return s;
  if (!g) return E3_ERR_INVALID_ARG;
  Ws w = kVariants[p->variant].ws(p, g);
  if (fwd_bytes) *fwd_bytes = 0;
  if (bwd_bytes) *bwd_bytes = w.t_bytes + w.dy_bytes;
  return E3_OK;
}

e3_status e3_conv_fwd(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* s,
                      float* m, void* ws, size_t ws_bytes, e3_stream stream) {
  (void)ws, (void)ws_bytes;
  e3_status st = check_plan(p);
  if (st != E3_OK) return st;
  if (!g) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!m || !aligned16(m) || !x || !aligned16(x))) return E3_ERR_INVALID_ARG;
  if (g->n_live > 0 && (!vec || !s || !aligned16(s))) return E3_ERR_INVALID_ARG;
  const VariantOps& v = kVariants[p->variant];
  return v.fwd[cpl_index(cpl_of(p))](p, g, x, vec, nullptr, s, m, 0, reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_conv_bwd(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* s,
                      const float* dm, float* dx, float* dvec, float* ds, void* ws, size_t ws_bytes,
                      e3_stream stream) {
  e3_status st = check_plan(p);
  if (st != E3_OK) return st;
  if (!g) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!x || !dm || !dx || !aligned16(x) || !aligned16(dm) || !aligned16(dx)))
    return E3_ERR_INVALID_ARG;
  if (g->n_edges > 0 && (!vec || !s || !ds || !dvec || !aligned16(s) || !aligned16(ds))) return E3_ERR_INVALID_ARG;
  const VariantOps& v = kVariants[p->variant];
  Ws w = v.ws(p, g);
  if (w.t_bytes + w.dy_bytes > 0 && (!ws || !aligned16(ws))) return E3_ERR_INVALID_ARG;
  if (ws_bytes < w.t_bytes + w.dy_bytes) return E3_ERR_WORKSPACE_TOO_SMALL;
  return v.bwd[cpl_index(cpl_of(p))](p, g, x, vec, nullptr, s, dm, dx, dvec, nullptr, ds, 0, ws,
                                     reinterpret_cast<hipStream_t>(stream));
}

}  // extern "C"

// ------------------------------------------------------------ no-allocation backward
// Scratch of e3_conv_bwd_noalloc: the per-edge x-cotangent partials and the
// per-wave harmonic-cotangent partials of the backward sweep, in a fixed
// array instead of a caller workspace.  Each device holds its own copy for the
// life of the process.  Host code never uses the array's name as an address:
// the device address comes from hipGetSymbolAddress, once per device.
constexpr size_t kNoAllocScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch`, looked up on the first call made
// with that device current.
e3_status scratch_of_current_device(void** out) {
  int dev = -1;
  E3_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) {
    g_last_error = "device ordinal beyond the no-allocation scratch table";
    return E3_ERR_UNSUPPORTED;
  }
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    E3_HIP(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
    if (!ptr) {
      g_last_error = "hipGetSymbolAddress returned no address for the scratch array";
      return E3_ERR_HIP;
    }
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return E3_OK;
}
}  // namespace

extern "C" {

e3_status e3_conv_bwd_noalloc(const e3_plan* p, const e3_graph* g, const float* x, const float* vec,
                              const float* s, const float* dm, float* dx, float* dvec, float* ds, e3_stream stream) {
  e3_status st = check_plan(p);
  if (st != E3_OK) return st;
  if (!g) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!x || !dm || !dx || !aligned16(x) || !aligned16(dm) || !aligned16(dx)))
    return E3_ERR_INVALID_ARG;
  if (g->n_edges > 0 && (!vec || !s || !ds || !dvec || !aligned16(s) || !aligned16(ds))) return E3_ERR_INVALID_ARG;
  const VariantOps& v = kVariants[p->variant];
  const Ws w = v.ws(p, g);
  if (w.t_bytes + w.dy_bytes > kNoAllocScratchBytes) {
    g_last_error = "the backward needs " + std::to_string(w.t_bytes + w.dy_bytes) +
                   " bytes of scratch; the no-allocation entry point has " + std::to_string(kNoAllocScratchBytes);
    return E3_ERR_WORKSPACE_TOO_SMALL;
  }
  void* ptr = nullptr;
  if ((st = scratch_of_current_device(&ptr)) != E3_OK) return st;
  // every scratch byte the kernels read is written earlier in the same call
  // (each live edge's partial rows and each wave's harmonic partials), so the
  // previous call's contents need no clearing
  return v.bwd[cpl_index(cpl_of(p))](p, g, x, vec, nullptr, s, dm, dx, dvec, nullptr, ds, 0, ptr,
                                     reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_conv_radial_workspace_size(const e3_plan* p, const e3_graph* g, int K, size_t* bwd_bytes) {
  e3_status st = check_plan(p);
  if (st != E3_OK) return st;
  if (!g || !bwd_bytes || K < 1 || K > kRadKMax) return E3_ERR_INVALID_ARG;
  *bwd_bytes = kVariants[p->variant].rws(p, g, K).total();
  return E3_OK;
}

e3_status e3_conv_fwd_radial(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* h,
                             const float* W, int K, float* m, e3_stream stream) {
  e3_status st = check_plan(p);
  if (st != E3_OK) return st;
  if (!g || K < 1 || K > kRadKMax) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!m || !aligned16(m) || !x || !aligned16(x) || !W || !aligned16(W))) return E3_ERR_INVALID_ARG;
  if (g->n_live > 0 && (!vec || !h)) return E3_ERR_INVALID_ARG;
  return kVariants[p->variant].rfwd(p, g, x, vec, h, W, K, m, reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_conv_bwd_radial(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* h,
                             const float* W, int K, const float* dm, float* dx, float* dvec, float* dh, float* dW,
                             void* ws, size_t ws_bytes, e3_stream stream) {
  e3_status st = check_plan(p);
  if (st != E3_OK) return st;
  if (!g || K < 1 || K > kRadKMax || !W || !aligned16(W) || !dW) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!x || !dm || !dx || !aligned16(x) || !aligned16(dm) || !aligned16(dx)))
    return E3_ERR_INVALID_ARG;
  if (g->n_edges > 0 && (!vec || !h || !dh || !dvec)) return E3_ERR_INVALID_ARG;
  const VariantOps& v = kVariants[p->variant];
  const RadWs w = v.rws(p, g, K);
  if (w.total() > 0 && (!ws || !aligned16(ws))) return E3_ERR_INVALID_ARG;
  if (ws_bytes < w.total()) return E3_ERR_WORKSPACE_TOO_SMALL;
  return v.rbwd(p, g, x, vec, h, W, K, dm, dx, dvec, dh, dW, ws, reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_conv_fwd_y(const e3_plan* p, const e3_graph* g, const float* x, const float* y, const float* s,
                        float* m, int accumulate, e3_stream stream) {
  e3_status st = check_plan(p);
  if (st != E3_OK) return st;
  if (!g) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!m || !aligned16(m) || !x || !aligned16(x))) return E3_ERR_INVALID_ARG;
  if (g->n_live > 0 && (!y || !s || !aligned16(s))) return E3_ERR_INVALID_ARG;
  const VariantOps& v = kVariants[p->variant];
  return v.fwd[cpl_index(cpl_of(p))](p, g, x, nullptr, y, s, m, accumulate != 0,
                                     reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_conv_bwd_y(const e3_plan* p, const e3_graph* g, const float* x, const float* y, const float* s,
                        const float* dm, float* dx, float* dy, float* ds, int accumulate, void* ws, size_t ws_bytes,
                        e3_stream stream) {
  e3_status st = check_plan(p);
  if (st != E3_OK) return st;
  if (!g) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!x || !dm || !aligned16(x) || !aligned16(dm) || (dx && !aligned16(dx))))
    return E3_ERR_INVALID_ARG;
  if (g->n_edges > 0 && (!y || !s || !aligned16(s) || (ds && !aligned16(ds)))) return E3_ERR_INVALID_ARG;
  const VariantOps& v = kVariants[p->variant];
  Ws w = v.ws(p, g);
  if (w.t_bytes + w.dy_bytes > 0 && (!ws || !aligned16(ws))) return E3_ERR_INVALID_ARG;
  if (ws_bytes < w.t_bytes + w.dy_bytes) return E3_ERR_WORKSPACE_TOO_SMALL;
  return v.bwd[cpl_index(cpl_of(p))](p, g, x, nullptr, y, s, dm, dx, nullptr, dy, ds,
                                     accumulate ? (kAccDx | kAccDy | kAccDs) : 0, ws,
                                     reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_conv_bwd2(const e3_plan* p, const e3_graph* g, const float* x, const float* y, const float* s,
                       const float* dm, const float* ddx, const float* ddy, const float* dds, float* gx, float* gy,
                       float* gs, float* gdm, void* ws, size_t ws_bytes, e3_stream stream) {
  e3_status st = check_plan(p);
  if (st != E3_OK) return st;
  if (!g) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!x || !dm || !ddx || !gx || !gdm || !aligned16(x) || !aligned16(dm) || !aligned16(ddx) ||
                         !aligned16(gx) || !aligned16(gdm)))
    return E3_ERR_INVALID_ARG;
  if (g->n_edges > 0 && (!y || !s || !ddy || !dds || !gy || !gs || !aligned16(s) || !aligned16(dds) ||
                         !aligned16(gs)))
    return E3_ERR_INVALID_ARG;
  const VariantOps& v = kVariants[p->variant];
  Ws w = v.ws(p, g);
  if (w.t_bytes + w.dy_bytes > 0 && (!ws || !aligned16(ws))) return E3_ERR_INVALID_ARG;
  if (ws_bytes < w.t_bytes + w.dy_bytes) return E3_ERR_WORKSPACE_TOO_SMALL;
  const int ci = cpl_index(cpl_of(p));
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  // ddm = conv(ddx, y, s) + conv(x, ddy, s) + conv(x, y, dds), in one pass
  if ((st = v.fwd3(p, g, x, ddx, y, ddy, s, dds, gdm, hs)) != E3_OK) return st;
  // gx, gy, gs in one sweep where the backward runs one channel per lane
  if (p->cpl_b == 1) return v.bwd3(p, g, x, ddx, y, ddy, s, dds, dm, gx, gy, gs, ws, hs);
  // (-, d_x y, d_x s) = conv_bwd(ddx, y, s, dm)
  if ((st = v.bwd[ci](p, g, ddx, nullptr, y, s, dm, nullptr, nullptr, gy, gs, 0, ws, hs)) != E3_OK) return st;
  // (d_y x, -, d_y s) = conv_bwd(x, ddy, s, dm)
  if ((st = v.bwd[ci](p, g, x, nullptr, ddy, s, dm, gx, nullptr, nullptr, gs, kAccDs, ws, hs)) != E3_OK) return st;
  // (d_s x, d_s y, -) = conv_bwd(x, y, dds, dm)
  return v.bwd[ci](p, g, x, nullptr, y, dds, dm, gx, nullptr, gy, nullptr, kAccDx | kAccDy, ws, hs);
}

}  // extern "C"

// ============================================================ linear mixing (host)
struct e3_linear {
  int d_in = 0, d_out = 0, c_in = 0, c_out = 0;
  int64_t nw = 0;
  std::vector<LinJob> fj, bj;   // forward jobs (output blocks), dx jobs (input blocks)
  std::vector<LinSrc> fs, bs;
  std::vector<LinPair> pairs;
  char* dev = nullptr;  // device copy of the tables (uploaded by e3_linear_create)
  int device = -1;      // the device that holds it
  size_t off_fj = 0, off_fs = 0, off_bj = 0, off_bs = 0, off_pairs = 0;
};

namespace {
// Device copy of the job and pair tables, on the current device (synchronous:
// called once, from e3_linear_create).
e3_status lin_upload(e3_linear* L) {
  size_t off = 0;
  auto place = [&](size_t bytes) { size_t o = off; off = align256(off + bytes); return o; };
  L->off_fj = place(L->fj.size() * sizeof(LinJob) + 1);
  L->off_fs = place(L->fs.size() * sizeof(LinSrc) + 1);
  L->off_bj = place(L->bj.size() * sizeof(LinJob) + 1);
  L->off_bs = place(L->bs.size() * sizeof(LinSrc) + 1);
  L->off_pairs = place(L->pairs.size() * sizeof(LinPair) + 1);
  std::vector<char> host(off, 0);
  auto put = [&](size_t o, const void* p, size_t b) { if (b) std::memcpy(host.data() + o, p, b); };
  put(L->off_fj, L->fj.data(), L->fj.size() * sizeof(LinJob));
  put(L->off_fs, L->fs.data(), L->fs.size() * sizeof(LinSrc));
  put(L->off_bj, L->bj.data(), L->bj.size() * sizeof(LinJob));
  put(L->off_bs, L->bs.data(), L->bs.size() * sizeof(LinSrc));
  put(L->off_pairs, L->pairs.data(), L->pairs.size() * sizeof(LinPair));
  E3_HIP(hipGetDevice(&L->device));
  char* d = nullptr;
  E3_HIP(hipMalloc(&d, off));
  const hipError_t e = hipMemcpy(d, host.data(), off, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    g_last_error = std::string("linear tables upload: ") + hipGetErrorString(e);
    (void)hipFree(d);
    return E3_ERR_HIP;
  }
  L->dev = d;
  return E3_OK;
}

// The tables live on the device current at creation; a call made with another
// device current is refused rather than reading another device's memory.
e3_status check_device(int device, const char* what) {
  int cur = -1;
  E3_HIP(hipGetDevice(&cur));
  if (cur != device) {
    g_last_error = std::string(what) + " was created on device " + std::to_string(device) +
                   ", called with device " + std::to_string(cur) + " current";
    return E3_ERR_INVALID_ARG;
  }
  return E3_OK;
}

e3_status lin_gemm(const std::vector<LinJob>& jobs, const LinJob* djobs, const LinSrc* dsrcs, const float* src,
                   const float* W, float* dst, int64_t n, int D_src, int C_src, int D_dst, int C_dst, int ldk, int ldc,
                   const char* name, hipStream_t st) {
  LinArgs a{};
  a.src = src, a.W = W, a.dst = dst, a.jobs = djobs, a.srcs = dsrcs, a.n = n;
  a.D_src = D_src, a.C_src = C_src, a.D_dst = D_dst, a.C_dst = C_dst, a.ldk = ldk, a.ldc = ldc;
  a.njobs = (int)jobs.size();
  a.slabs = (C_dst + kWave - 1) / kWave;
  int64_t u = 0;
  for (size_t j = 0; j < jobs.size(); ++j) {
    a.first[j] = (int)u;
    u += (n * jobs[j].R + 16 * kLinRT - 1) / (16 * kLinRT) * a.slabs;
  }
  a.first[jobs.size()] = (int)u;
  if (u == 0) return E3_OK;
  if (u > 0x7fffffff) return E3_ERR_INVALID_ARG;
  TimedLaunch t_(name, st);
  if (ldc == 1 && C_dst % 4 == 0 && aligned16(W) && E3_LIN_V4)
    hipLaunchKernelGGL((k_lin_gemm<kLinRT, true>), dim3((unsigned)u), dim3(kWave), 0, st, a);
  else
    hipLaunchKernelGGL((k_lin_gemm<kLinRT, false>), dim3((unsigned)u), dim3(kWave), 0, st, a);
  E3_HIP(hipGetLastError());
  return E3_OK;
}

// dW partials, then W transposed slice by slice (read by dx along rows)
size_t lin_ws_dwp(const e3_linear* L) {
  return align256((size_t)L->pairs.size() * kLinChunks * L->c_in * L->c_out * sizeof(float));
}
size_t lin_ws(const e3_linear* L) { return lin_ws_dwp(L) + align256((size_t)L->nw * sizeof(float)); }
}  // namespace

extern "C" {

e3_status e3_linear_create(const char* irreps_in, const char* irreps_out, e3_linear** out) {
  if (!irreps_in || !irreps_out || !out) return E3_ERR_INVALID_ARG;
  *out = nullptr;
  std::vector<e3b::Block> bi, bo;
  std::string err;
  if (!e3b::parse_irreps(irreps_in, bi, err) || !e3b::parse_irreps(irreps_out, bo, err)) {
    g_last_error = err;
    return E3_ERR_INVALID_ARG;
  }
  const int c_in = bi[0].mul, c_out = bo[0].mul;
  for (const auto& b : bi)
    if (b.mul != c_in) return E3_ERR_INVALID_ARG;
  for (const auto& b : bo)
    if (b.mul != c_out) return E3_ERR_INVALID_ARG;
  if (c_in % 16 || c_out % 16 || c_in > 4096 || c_out > 4096) {
    g_last_error = "linear mixing needs multiplicities that are multiples of 16 (at most 4096)";
    return E3_ERR_UNSUPPORTED;
  }
  if ((int)bi.size() > kLinMaxJobs || (int)bo.size() > kLinMaxJobs) {
    g_last_error = "linear mixing supports at most 64 blocks per side";
    return E3_ERR_UNSUPPORTED;
  }
  e3_linear* L = new (std::nothrow) e3_linear();
  if (!L) return E3_ERR_ALLOC;
  L->c_in = c_in, L->c_out = c_out;
  std::vector<int> irow(bi.size()), orow(bo.size());
  for (size_t i = 0; i < bi.size(); ++i) irow[i] = L->d_in, L->d_in += 2 * bi[i].l + 1;
  for (size_t o = 0; o < bo.size(); ++o) orow[o] = L->d_out, L->d_out += 2 * bo[o].l + 1;
  // forward: one job per output block, sources = input blocks of its type, in order
  std::vector<std::vector<std::pair<int, int64_t>>> feeds(bi.size());  // input -> (output, W offset)
  int64_t woff = 0;
  for (size_t o = 0; o < bo.size(); ++o) {
    LinJob j{2 * bo[o].l + 1, orow[o], (int)L->fs.size(), 0};
    for (size_t i = 0; i < bi.size(); ++i)
      if (bi[i].l == bo[o].l && bi[i].p == bo[o].p) {
        L->fs.push_back(LinSrc{irow[i], 0, woff});
        L->pairs.push_back(LinPair{j.R, irow[i], orow[o], 0, woff});
        feeds[i].push_back({(int)o, woff});
        woff += (int64_t)c_in * c_out;
        ++j.nsrc;
      }
    L->fj.push_back(j);
  }
  L->nw = woff;
  // dx: one job per input block, sources = the output blocks it feeds (W read transposed)
  for (size_t i = 0; i < bi.size(); ++i) {
    LinJob j{2 * bi[i].l + 1, irow[i], (int)L->bs.size(), (int)feeds[i].size()};
    for (auto& f : feeds[i]) L->bs.push_back(LinSrc{orow[f.first], 0, f.second});
    L->bj.push_back(j);
  }
  const e3_status st = lin_upload(L);
  if (st != E3_OK) {
    delete L;
    return st;
  }
  *out = L;
  return E3_OK;
}

e3_status e3_linear_query(const e3_linear* L, int64_t* n_weights, int* d_in, int* d_out, int* c_in, int* c_out) {
  if (!L) return E3_ERR_INVALID_ARG;
  if (n_weights) *n_weights = L->nw;
  if (d_in) *d_in = L->d_in;
  if (d_out) *d_out = L->d_out;
  if (c_in) *c_in = L->c_in;
  if (c_out) *c_out = L->c_out;
  return E3_OK;
}

e3_status e3_linear_destroy(e3_linear* L) {
  if (!L) return E3_OK;
  if (L->dev) (void)hipFree(L->dev);
  delete L;
  return E3_OK;
}

e3_status e3_linear_fwd(e3_linear* L, const float* x, const float* W, float* out, int64_t n, e3_stream stream) {
  if (!L || n < 0) return E3_ERR_INVALID_ARG;
  if (n == 0) return E3_OK;
  if (!x || !W || !out || !aligned16(x) || !aligned16(out)) return E3_ERR_INVALID_ARG;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  e3_status s = check_device(L->device, "linear mixing handle");
  if (s != E3_OK) return s;
  return lin_gemm(L->fj, reinterpret_cast<const LinJob*>(L->dev + L->off_fj),
                  reinterpret_cast<const LinSrc*>(L->dev + L->off_fs), x, W, out, n, L->d_in, L->c_in, L->d_out,
                  L->c_out, L->c_out, 1, "linear_fwd", st);
}

e3_status e3_linear_workspace_size(const e3_linear* L, size_t* bwd_bytes) {
  if (!L || !bwd_bytes) return E3_ERR_INVALID_ARG;
  *bwd_bytes = lin_ws(L);
  return E3_OK;
}

e3_status e3_linear_bwd(e3_linear* L, const float* x, const float* W, const float* dout, float* dx, float* dW,
                        void* ws, size_t ws_bytes, int64_t n, e3_stream stream) {
  if (!L || n < 0) return E3_ERR_INVALID_ARG;
  if (!W || !dW || (n > 0 && (!x || !dout || !dx || !aligned16(x) || !aligned16(dout) || !aligned16(dx))))
    return E3_ERR_INVALID_ARG;
  if (ws_bytes < lin_ws(L)) return E3_ERR_WORKSPACE_TOO_SMALL;
  if (lin_ws(L) > 0 && (!ws || !aligned16(ws))) return E3_ERR_INVALID_ARG;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  e3_status s = check_device(L->device, "linear mixing handle");
  if (s != E3_OK) return s;
  const LinPair* dp = reinterpret_cast<const LinPair*>(L->dev + L->off_pairs);
  if (n > 0) {
    // slices of Wt sit at the same offsets as those of W (pair order)
    float* Wt = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + lin_ws_dwp(L));
    if (!L->pairs.empty()) {
      TimedLaunch t_("linear_bwd_transpose", st);
      hipLaunchKernelGGL(k_lin_transpose, dim3(blocks_for(L->nw, 256)), dim3(256), 0, st, W, dp, Wt,
                         (int)L->pairs.size(), L->c_in, L->c_out);
      E3_HIP(hipGetLastError());
    }
    s = lin_gemm(L->bj, reinterpret_cast<const LinJob*>(L->dev + L->off_bj),
                 reinterpret_cast<const LinSrc*>(L->dev + L->off_bs), dout, Wt, dx, n, L->d_out, L->c_out, L->d_in,
                 L->c_in, L->c_in, 1, "linear_bwd_dx", st);
    if (s != E3_OK) return s;
  }
  if (L->pairs.empty()) return E3_OK;
  float* dWp = reinterpret_cast<float*>(ws);
  LinDwArgs a{};
  a.x = x, a.dout = dout, a.dWp = dWp, a.pairs = dp, a.n = n;
  a.D_in = L->d_in, a.C_in = L->c_in, a.D_out = L->d_out, a.C_out = L->c_out;
  a.ktiles = (L->c_in + 63) / 64, a.jtiles = (L->c_out + 63) / 64;
  {
    TimedLaunch t_("linear_bwd_dw", st);
    const int64_t units = (int64_t)L->pairs.size() * kLinChunks * a.ktiles * a.jtiles;
    hipLaunchKernelGGL(k_lin_dw, dim3((unsigned)units), dim3(kWave), 0, st, a);
    E3_HIP(hipGetLastError());
  }
  {
    TimedLaunch t_("linear_bwd_dw_sum", st);
    const int64_t per = (int64_t)L->c_in * L->c_out;
    hipLaunchKernelGGL(k_lin_dw_sum, dim3(blocks_for(per * (int64_t)L->pairs.size(), 256)), dim3(256), 0, st, dWp, dp,
                       dW, (int)L->pairs.size(), per);
    E3_HIP(hipGetLastError());
  }
  return E3_OK;
}

}  // extern "C"

// ============================================================ generic records (host)
struct e3_tpg {
  int d_x = 0, d_y = 0, d_z = 0, ypc = 0;
  // record tables: forward (out z, A x, B y), dx (out x, A dz, B y), dy (out y, A x, B dz)
  struct Table {
    std::vector<int> seg;
    std::vector<TpgRec> recs;
    std::vector<TpgRec64> recs64;
    size_t off_seg = 0, off_recs = 0, off_recs64 = 0;
  } t[3];
  char* dev = nullptr;  // device copy of the tables (uploaded by e3_tpg_create)
  int device = -1;      // the device that holds it
};

namespace {
e3_tpg::Table tpg_table(int d_out, const std::vector<std::array<int, 3>>& key, const std::vector<double>& val) {
  // key = (out, a, b); stable order by (out, a, b)
  std::vector<size_t> ord(key.size());
  for (size_t i = 0; i < ord.size(); ++i) ord[i] = i;
  std::stable_sort(ord.begin(), ord.end(), [&](size_t u, size_t v) { return key[u] < key[v]; });
  e3_tpg::Table T;
  T.seg.assign(d_out + 1, 0);
  for (size_t i : ord) {
    T.recs.push_back(TpgRec{key[i][1], key[i][2], (float)val[i], 0});
    T.recs64.push_back(TpgRec64{key[i][1], key[i][2], val[i]});
    ++T.seg[key[i][0] + 1];
  }
  for (int o = 0; o < d_out; ++o) T.seg[o + 1] += T.seg[o];
  return T;
}

// Device copy of the record tables, on the current device (synchronous:
// called once, from e3_tpg_create).
e3_status tpg_upload(e3_tpg* G) {
  size_t off = 0;
  for (auto& T : G->t) {
    T.off_seg = off;
    off = align256(off + T.seg.size() * sizeof(int));
    T.off_recs = off;
    off = align256(off + T.recs.size() * sizeof(TpgRec) + 1);
    T.off_recs64 = off;
    off = align256(off + T.recs64.size() * sizeof(TpgRec64) + 1);
  }
  std::vector<char> host(off, 0);
  for (auto& T : G->t) {
    std::memcpy(host.data() + T.off_seg, T.seg.data(), T.seg.size() * sizeof(int));
    if (!T.recs.empty()) std::memcpy(host.data() + T.off_recs, T.recs.data(), T.recs.size() * sizeof(TpgRec));
    if (!T.recs64.empty())
      std::memcpy(host.data() + T.off_recs64, T.recs64.data(), T.recs64.size() * sizeof(TpgRec64));
  }
  E3_HIP(hipGetDevice(&G->device));
  char* d = nullptr;
  E3_HIP(hipMalloc(&d, off));
  const hipError_t e = hipMemcpy(d, host.data(), off, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    g_last_error = std::string("record tables upload: ") + hipGetErrorString(e);
    (void)hipFree(d);
    return E3_ERR_HIP;
  }
  G->dev = d;
  return E3_OK;
}

size_t tpg_lds(int dA, int dB, int dout, bool bsh, bool red, size_t elem = sizeof(float), int rb = 1) {
  return ((size_t)dA * rb * kWave + (bsh ? (((size_t)dB * rb + 3) & ~3) : (size_t)dB * rb * kWave) +
          (red ? (size_t)dout * rb * kWave : 0)) *
         elem;
}
constexpr size_t kTpgMaxLds = 64 * 1024;

template <class T>
e3_status tpg_run(const e3_tpg* G, int which, const T* A, int dA, const T* B, int dB, bool bsh, T* out, T* part,
                  bool red, int64_t rows, int C, const char* name, hipStream_t st) {
  const e3_tpg::Table& Tb = G->t[which];
  TpgArgs<T> a{};
  a.A = A, a.B = B, a.out = out, a.part = part;
  a.seg = reinterpret_cast<const int*>(G->dev + Tb.off_seg);
  a.recs = reinterpret_cast<decltype(a.recs)>(G->dev + (sizeof(T) == 8 ? Tb.off_recs64 : Tb.off_recs));
  a.rows = rows, a.C = C, a.nslab = (C + kWave - 1) / kWave, a.dA = dA, a.dB = dB;
  a.dout = (int)Tb.seg.size() - 1;
  // rows per wave: the most of 4, 2, 1 whose staging fits the LDS limit
  int rb = 4;
  while (rb > 1 && tpg_lds(dA, dB, a.dout, bsh, red, sizeof(T), rb) > kTpgMaxLds) rb /= 2;
  const size_t lds = tpg_lds(dA, dB, a.dout, bsh, red, sizeof(T), rb);
  if (lds > kTpgMaxLds) return E3_ERR_UNSUPPORTED;
  // operand blocks are addressed with 32-bit byte offsets
  if ((int64_t)rb * std::max(dA, dB) * C * (int64_t)sizeof(T) > 0x7fffffff) return E3_ERR_INVALID_ARG;
  const int64_t grid = tile_grid(false, rows, rb, a.nslab);
  if (grid > 0x7fffffff) return E3_ERR_INVALID_ARG;
  TimedLaunch t_(name, st);
  auto go = [&](auto RBc) {
    constexpr int R = decltype(RBc)::value;
    if (bsh && red)
      hipLaunchKernelGGL((k_tpg<T, true, true, R>), dim3((unsigned)grid), dim3(kWave), lds, st, a);
    else if (bsh)
      hipLaunchKernelGGL((k_tpg<T, true, false, R>), dim3((unsigned)grid), dim3(kWave), lds, st, a);
    else if (red)
      hipLaunchKernelGGL((k_tpg<T, false, true, R>), dim3((unsigned)grid), dim3(kWave), lds, st, a);
    else
      hipLaunchKernelGGL((k_tpg<T, false, false, R>), dim3((unsigned)grid), dim3(kWave), lds, st, a);
  };
  if (rb == 4)
    go(std::integral_constant<int, 4>{});
  else if (rb == 2)
    go(std::integral_constant<int, 2>{});
  else
    go(std::integral_constant<int, 1>{});
  E3_HIP(hipGetLastError());
  return E3_OK;
}
}  // namespace

extern "C" {

e3_status e3_tpg_create(int d_x, int d_y, int d_z, int64_t nnz, const int32_t* i0, const int32_t* i1,
                        const int32_t* i2, const double* val, int y_per_channel, e3_tpg** out) {
  if (!out) return E3_ERR_INVALID_ARG;
  *out = nullptr;
  if (d_x < 1 || d_y < 1 || d_z < 1 || nnz < 0 || nnz > (1 << 24) || (nnz > 0 && (!i0 || !i1 || !i2 || !val)))
    return E3_ERR_INVALID_ARG;
  for (int64_t k = 0; k < nnz; ++k)
    if (i0[k] < 0 || i0[k] >= d_z || i1[k] < 0 || i1[k] >= d_x || i2[k] < 0 || i2[k] >= d_y)
      return E3_ERR_INDEX_OUT_OF_RANGE;
  const bool bsh = !y_per_channel;
  if (tpg_lds(d_x, d_y, d_z, bsh, false) > kTpgMaxLds || tpg_lds(d_z, d_y, d_x, bsh, false) > kTpgMaxLds ||
      tpg_lds(d_x, d_z, d_y, false, bsh) > kTpgMaxLds) {
    g_last_error = "record tensor product: operand rows do not fit the 64 KiB staging limit";
    return E3_ERR_UNSUPPORTED;
  }
  e3_tpg* G = new (std::nothrow) e3_tpg();
  if (!G) return E3_ERR_ALLOC;
  G->d_x = d_x, G->d_y = d_y, G->d_z = d_z, G->ypc = y_per_channel ? 1 : 0;
  std::vector<std::array<int, 3>> kf(nnz), kx(nnz), ky(nnz);
  std::vector<double> v(val, val + nnz);
  for (int64_t k = 0; k < nnz; ++k) {
    kf[k] = {i0[k], i1[k], i2[k]};  // z[i0] from x[i1], y[i2]
    kx[k] = {i1[k], i0[k], i2[k]};  // dx[i1] from dz[i0], y[i2]   (records (i1, i2, i0) of eq. tp-bwd)
    ky[k] = {i2[k], i1[k], i0[k]};  // dy[i2] from x[i1], dz[i0]   (records (i2, i1, i0))
  }
  G->t[0] = tpg_table(d_z, kf, v);
  G->t[1] = tpg_table(d_x, kx, v);
  G->t[2] = tpg_table(d_y, ky, v);
  const e3_status st = tpg_upload(G);
  if (st != E3_OK) {
    delete G;
    return st;
  }
  *out = G;
  return E3_OK;
}

e3_status e3_tpg_destroy(e3_tpg* G) {
  if (!G) return E3_OK;
  if (G->dev) (void)hipFree(G->dev);
  delete G;
  return E3_OK;
}

}  // extern "C"

namespace {
template <class T>
e3_status tpg_fwd(e3_tpg* G, const T* x, const T* y, T* z, int64_t rows, int C, hipStream_t st) {
  if (!G || rows < 0 || C < 1) return E3_ERR_INVALID_ARG;
  if (rows == 0) return E3_OK;
  if (!x || !y || !z) return E3_ERR_INVALID_ARG;
  e3_status s = check_device(G->device, "record tensor-product handle");
  if (s != E3_OK) return s;
  return tpg_run<T>(G, 0, x, G->d_x, y, G->d_y, !G->ypc, z, nullptr, false, rows, C,
                    sizeof(T) == 8 ? "tpg_fwd_f64" : "tpg_fwd", st);
}

size_t tpg_ws(const e3_tpg* G, int64_t rows, int C, size_t elem) {
  return G->ypc ? 0 : align256((size_t)rows * ((C + kWave - 1) / kWave) * G->d_y * elem);
}

template <class T>
e3_status tpg_bwd(e3_tpg* G, const T* x, const T* y, const T* dz, T* dx, T* dy, void* ws, size_t ws_bytes,
                  int64_t rows, int C, hipStream_t st) {
  if (!G || rows < 0 || C < 1) return E3_ERR_INVALID_ARG;
  if (rows == 0) return E3_OK;
  if (!x || !y || !dz || !dx || !dy) return E3_ERR_INVALID_ARG;
  const size_t need = tpg_ws(G, rows, C, sizeof(T));
  if (ws_bytes < need) return E3_ERR_WORKSPACE_TOO_SMALL;
  if (need > 0 && !ws) return E3_ERR_INVALID_ARG;
  e3_status s = check_device(G->device, "record tensor-product handle");
  if (s != E3_OK) return s;
  const bool f64 = sizeof(T) == 8;
  // dx = tensor_product(C^{i1}_{i2 i0}, y, dz)
  if ((s = tpg_run<T>(G, 1, dz, G->d_z, y, G->d_y, !G->ypc, dx, nullptr, false, rows, C,
                      f64 ? "tpg_bwd_dx_f64" : "tpg_bwd_dx", st)) != E3_OK)
    return s;
  // dy = tensor_product(C^{i2}_{i1 i0}, x, dz), summed over the channels when y is shared
  if (G->ypc)
    return tpg_run<T>(G, 2, x, G->d_x, dz, G->d_z, false, dy, nullptr, false, rows, C,
                      f64 ? "tpg_bwd_dy_f64" : "tpg_bwd_dy", st);
  T* part = reinterpret_cast<T*>(ws);
  if ((s = tpg_run<T>(G, 2, x, G->d_x, dz, G->d_z, false, nullptr, part, true, rows, C,
                      f64 ? "tpg_bwd_dy_f64" : "tpg_bwd_dy", st)) != E3_OK)
    return s;
  TimedLaunch t_(f64 ? "tpg_bwd_dy_sum_f64" : "tpg_bwd_dy_sum", st);
  hipLaunchKernelGGL(k_tpg_sum<T>, dim3(blocks_for(rows * G->d_y, 256)), dim3(256), 0, st, part, dy, rows,
                     (C + kWave - 1) / kWave, G->d_y);
  E3_HIP(hipGetLastError());
  return E3_OK;
}
}  // namespace

extern "C" {

e3_status e3_tpg_fwd(e3_tpg* G, const float* x, const float* y, float* z, int64_t rows, int C, e3_stream stream) {
  return tpg_fwd<float>(G, x, y, z, rows, C, reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_tpg_fwd_f64(e3_tpg* G, const double* x, const double* y, double* z, int64_t rows, int C,
                         e3_stream stream) {
  return tpg_fwd<double>(G, x, y, z, rows, C, reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_tpg_workspace_size(const e3_tpg* G, int64_t rows, int C, size_t* bwd_bytes) {
  if (!G || rows < 0 || C < 1 || !bwd_bytes) return E3_ERR_INVALID_ARG;
  *bwd_bytes = tpg_ws(G, rows, C, sizeof(double));  // enough for either precision
  return E3_OK;
}

e3_status e3_tpg_bwd(e3_tpg* G, const float* x, const float* y, const float* dz, float* dx, float* dy, void* ws,
                     size_t ws_bytes, int64_t rows, int C, e3_stream stream) {
  return tpg_bwd<float>(G, x, y, dz, dx, dy, ws, ws_bytes, rows, C, reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_tpg_bwd_f64(e3_tpg* G, const double* x, const double* y, const double* dz, double* dx, double* dy,
                         void* ws, size_t ws_bytes, int64_t rows, int C, e3_stream stream) {
  return tpg_bwd<double>(G, x, y, dz, dx, dy, ws, ws_bytes, rows, C, reinterpret_cast<hipStream_t>(stream));
}

}  // extern "C"

// ============================================================ streaming probe
// Instrumentation: the bandwidth HBM sustains for a given read:write mix, with
// the load and store instructions of the sweeps (buffer loads and stores of
// WB bytes per lane at a per-lane offset, with or without the non-temporal
// bit).  Step s reads RU contiguous units of the source and writes WU
// contiguous units of the destination (a unit is 64 lanes x WB bytes), so the
// traffic mix is RU:WU; waves take steps in grid-stride order, so neighbouring
// waves stream neighbouring memory.
// Written only if a wave's sum of loaded values is 3e38, i.e. never for the
// probe's data; its device address is a kernel argument, so that the compiler
// cannot prove the loads feeding that sum unused.
static __device__ __align__(256) float probe_sink[4096];

namespace {

template <int WB, int AUX>
__device__ __forceinline__ float probe_load(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  if constexpr (WB == 4) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, AUX));
  } else if constexpr (WB == 8) {
    const f2v t = __builtin_bit_cast(f2v, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, AUX));
    return t.x + t.y;
  } else {
    const f4v t = __builtin_bit_cast(f4v, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, AUX));
    return (t.x + t.y) + (t.z + t.w);
  }
}

template <int WB, int AUX>
__device__ __forceinline__ void probe_store(__amdgpu_buffer_rsrc_t r, int voff, int soff, float v) {
  const unsigned u = __builtin_bit_cast(unsigned, v);
  if constexpr (WB == 4) {
    __builtin_amdgcn_raw_buffer_store_b32(u, r, voff, soff, AUX);
  } else if constexpr (WB == 8) {
    typedef unsigned u2v __attribute__((ext_vector_type(2)));
    __builtin_amdgcn_raw_buffer_store_b64(u2v{u, u}, r, voff, soff, AUX);
  } else {
    typedef unsigned u4v __attribute__((ext_vector_type(4)));
    __builtin_amdgcn_raw_buffer_store_b128(u4v{u, u, u, u}, r, voff, soff, AUX);
  }
}

// Compiled probe shapes (read units, write units, bytes per lane): all loads
// of a step are issued before any is used, as the sweeps issue a row's loads.
#define E3_PROBE_SHAPES(X) \
  X(16, 0, 16) X(16, 0, 8) X(16, 0, 4) X(0, 16, 16) X(0, 16, 8) X(0, 16, 4) X(8, 8, 16) X(14, 1, 8) \
  X(14, 16, 4) X(2, 6, 8) X(8, 2, 8)

template <int WB, int RU, int WU, int LA, int SA>
__global__ __launch_bounds__(256) void k_probe(const char* __restrict__ src, char* __restrict__ dst,
                                               int64_t n_steps, float* __restrict__ sink) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t nw = (int64_t)gridDim.x * (blockDim.x / kWave);
  // wave index, uniform across the wave (buffer descriptors need scalar bases)
  const int64_t w0 = (int64_t)blockIdx.x * (blockDim.x / kWave) + uniform((int)(threadIdx.x / kWave));
  constexpr int unit = kWave * WB;
  float acc = 0.0f;
  for (int64_t s = w0; s < n_steps; s += nw) {
    if constexpr (RU > 0) {
      const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<char*>(src) + s * RU * unit, (short)0, RU * unit, 0x00020000);
      float v[RU];
#pragma unroll
      for (int u = 0; u < RU; ++u) v[u] = probe_load<WB, LA>(r, lane * WB, u * unit);
#pragma unroll
      for (int u = 0; u < RU; ++u) acc += v[u];
    }
    if constexpr (WU > 0) {
      const __amdgpu_buffer_rsrc_t r =
          __builtin_amdgcn_make_buffer_rsrc(dst + s * WU * unit, (short)0, WU * unit, 0x00020000);
      const float val = (float)(s & 1023);
#pragma unroll
      for (int u = 0; u < WU; ++u) probe_store<WB, SA>(r, lane * WB, u * unit, val);
    }
  }
  // keeps the loads: never true for finite data below 1e30
  if (acc == 3.0e38f) sink[w0 & 4095] = acc;
}

template <int WB, int RU, int WU>
void probe_launch(const char* src, char* dst, int64_t steps, unsigned flags, int blocks, float* sink,
                  hipStream_t st) {
  const bool nl = flags & 1u, ns = flags & 2u;
  if (nl && ns)
    hipLaunchKernelGGL((k_probe<WB, RU, WU, kNT, kST>), dim3(blocks), dim3(256), 0, st, src, dst, steps, sink);
  else if (nl)
    hipLaunchKernelGGL((k_probe<WB, RU, WU, kNT, 0>), dim3(blocks), dim3(256), 0, st, src, dst, steps, sink);
  else if (ns)
    hipLaunchKernelGGL((k_probe<WB, RU, WU, 0, kST>), dim3(blocks), dim3(256), 0, st, src, dst, steps, sink);
  else
    hipLaunchKernelGGL((k_probe<WB, RU, WU, 0, 0>), dim3(blocks), dim3(256), 0, st, src, dst, steps, sink);
}

bool probe_shape_supported(int ru, int wu, int width) {
#define E3_PROBE_IS(R, W, B) if (ru == R && wu == W && width == B) return true;
  E3_PROBE_SHAPES(E3_PROBE_IS)
#undef E3_PROBE_IS
  return false;
}

std::mutex g_sink_mu;
float* g_sink_ptr[64] = {};

// The current device's copy of probe_sink (looked up once per device).
e3_status sink_of_current_device(float** out) {
  int dev = -1;
  E3_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) return E3_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lk(g_sink_mu);
  if (!g_sink_ptr[dev]) {
    void* ptr = nullptr;
    E3_HIP(hipGetSymbolAddress(&ptr, HIP_SYMBOL(probe_sink)));
    g_sink_ptr[dev] = static_cast<float*>(ptr);
  }
  *out = g_sink_ptr[dev];
  return *out ? E3_OK : E3_ERR_HIP;
}
}  // namespace

extern "C" e3_status e3_probe_stream(const void* src, size_t src_bytes, void* dst, size_t dst_bytes,
                                     int read_units, int write_units, int width, unsigned flags,
                                     size_t* bytes_read, size_t* bytes_written, e3_stream stream) {
  if (read_units < 0 || write_units < 0 || read_units + write_units == 0 ||
      (width != 4 && width != 8 && width != 16) || flags > 3u || !bytes_read || !bytes_written)
    return E3_ERR_INVALID_ARG;
  if ((read_units > 0 && (!src || !aligned16(src))) || (write_units > 0 && (!dst || !aligned16(dst))))
    return E3_ERR_INVALID_ARG;
  if (!probe_shape_supported(read_units, write_units, width)) {
    g_last_error = "probe shape not compiled (see E3_PROBE_SHAPES)";
    return E3_ERR_UNSUPPORTED;
  }
  const int64_t unit = (int64_t)kWave * width;
  int64_t steps = INT64_MAX;
  if (read_units > 0) steps = std::min<int64_t>(steps, (int64_t)(src_bytes / (size_t)(unit * read_units)));
  if (write_units > 0) steps = std::min<int64_t>(steps, (int64_t)(dst_bytes / (size_t)(unit * write_units)));
  *bytes_read = (size_t)(steps * unit * read_units);
  *bytes_written = (size_t)(steps * unit * write_units);
  if (steps == 0) return E3_OK;
  // eight waves per SIMD on every compute unit, or fewer when there is less work
  const int blocks = (int)std::min<int64_t>((steps + 3) / 4, 2048);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const char* s = static_cast<const char*>(src);
  char* d = static_cast<char*>(dst);
  float* sink = nullptr;
  const e3_status ss = sink_of_current_device(&sink);
  if (ss != E3_OK) return ss;
  TimedLaunch t_("probe_stream", st);
#define E3_PROBE_GO(R, W, B) \
  if (read_units == R && write_units == W && width == B) probe_launch<B, R, W>(s, d, steps, flags, blocks, sink, st);
  E3_PROBE_SHAPES(E3_PROBE_GO)
#undef E3_PROBE_GO
  E3_HIP(hipGetLastError());
  return E3_OK;
}
