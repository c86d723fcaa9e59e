// e3mi: shared part of every translation unit of the library -- the row
// access helpers, the kernels that are templated on the irreps variant, the
// handle structures and the host launchers of each variant.  The variant
// units (one per compiled irreps layout) instantiate the launchers for their
// layout; the core unit (e3mi.hip) holds everything else and the C ABI.
#pragma once
#include <hip/hip_runtime.h>

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
// Three-term forward of the double backward: 1 runs the waves of two channel
// slabs of one (receiver, group) in one workgroup, sharing the staged
// pre-contractions (2.4% faster at equal batches); 0 gives every slab its own
// workgroup.
#ifndef E3_FWD3_PAIR
#define E3_FWD3_PAIR 1
#endif
// Edges per staged batch of a slab pair (at most 64): 16 measured 3.7% faster
// than 8 and 12, 24 and 32 slower (fewer workgroups fit the LDS).
#ifndef E3_FWD3_BATCH2
#define E3_FWD3_BATCH2 16
#endif
static_assert(E3_FWD3_BATCH2 >= 1 && E3_FWD3_BATCH2 <= 64, "one lane per edge of a batch");
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


// ------------------------------------------------------------ shared state
// Defined once, in the core unit.
extern thread_local std::string g_last_error;
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
extern Timing g_timing;

namespace {


// ------------------------------------------------------------ launch timing
// When enabled, every kernel launch of the library is bracketed by two HIP
// events recorded on the caller's stream; e3_timing_read() resolves them into
// per-kernel summed durations.  Off by default (no events recorded).

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

// Row strides and harmonic-partial slots: the variant's own for a compiled
// layout, the whole layout's (given at run time) for a single-block kind.
template <class V, class A>
__device__ __forceinline__ int x_rows(const A& a) {
  if constexpr (V::RT) return a.xr;
  else return V::D_IN;
}
template <class V, class A>
__device__ __forceinline__ int p_rows(const A& a) {
  if constexpr (V::RT) return a.pr;
  else return V::NP;
}
template <class V, class A>
__device__ __forceinline__ int o_rows(const A& a) {
  if constexpr (V::RT) return a.orr;
  else return V::D_OUT;
}
template <class V, int G, class A>
__device__ __forceinline__ int64_t dy_group(const A& a, int64_t pos) {
  if constexpr (V::RT) return pos * a.ng + a.g0 + G;
  else return pos * V::NBG + G;
}

// Row strides of a single-block kind's tensor product inside a larger layout
// (unused by compiled layouts).
struct TpStr {
  int xr, pr, orr;
};

// ------------------------------------------------------------ tensor product
constexpr int kTpRows = 8;  // rows whose pre-contraction is staged per LDS batch

template <class V, int CPL>
__global__ __launch_bounds__(kWave) void k_tp(const float* __restrict__ x, const float* __restrict__ y,
                                              const float* __restrict__ w, float* __restrict__ z, int64_t rows,
                                              int C, int nslab, TpStr ts) {
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
    const RowBuf xb = row_buf(x + r * x_rows<V>(ts) * C, (int64_t)V::D_IN * C * 4, q, C);
    const RowBuf wb = row_buf(w + r * p_rows<V>(ts) * C, (int64_t)V::NP * C * 4, q, C);
    const RowBuf zb = row_buf(z + r * o_rows<V>(ts) * C, (int64_t)V::D_OUT * C * 4, q, C);
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
  int xr, pr, orr, ng, g0;  // a single-block kind inside a larger layout (as in ConvArgs)
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
      const RowBuf xb = row_buf(a.x + r * x_rows<V>(a) * C, (int64_t)V::D_IN * C * 4, q, C);
      const RowBuf wb = row_buf(a.w + r * p_rows<V>(a) * C, (int64_t)V::NP * C * 4, q, C);
      const RowBuf zb = row_buf(a.dz + r * o_rows<V>(a) * C, (int64_t)V::D_OUT * C * 4, q, C);
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
      const RowBuf dwb = row_buf(a.dw + r * p_rows<V>(a) * C, (int64_t)V::NP * C * 4, q, C);
      auto st = [&](int pl, const float (&v)[CPL]) { bst<CPL, kST>(dwb, B::PATH[pl], v); };
      float dyl[V::D_SH];
#pragma unroll
      for (int i = 0; i < V::D_SH; ++i) dyl[i] = 0.0f;
      B::template edge<false, CPL>(sA + j * B::NA, Yv, xv, wv, dzv, t, dyl, st);
#pragma unroll
      for (int i = 0; i < V::D_SH; ++i) dy[i] = dyl[i];
      const RowBuf dxb = row_buf(a.dx + r * x_rows<V>(a) * C, (int64_t)V::D_IN * C * 4, q, C);
#pragma unroll
      for (int i = 0; i < B::NXR; ++i) bst<CPL, kST>(dxb, B::XROW[i], t[i]);
    }
    const float tot = wave_reduce16(dy, lane);
    if ((lane & 3) == 0) a.DY[(dy_group<V, G>(a, r) * a.nslab + sl) * 16 + (lane >> 2)] = tot;
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
  int sw;  // three-term forward: slab waves per workgroup (1, or 2 sharing the staged A and A2)
  int fb;  // three-term forward: edges per staged batch
  // a single-block kind (V::RT) inside a larger layout: rows of the whole
  // layout per node of x / dx / T slot, per edge of s / ds, per node of m /
  // dm, and its harmonic-partial groups (all of them, and this block's first)
  int xr, pr, orr, ng, g0;
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
        const RowBuf xb_ = row_buf(a.x + snd * x_rows<V>(a) * C, (int64_t)V::D_IN * C * 4, q, C);
        const RowBuf sb_ = row_buf(a.s + e * p_rows<V>(a) * C, (int64_t)V::NP * C * 4, q, C);
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
    const RowBuf mb = row_buf(a.m + (int64_t)b * o_rows<V>(a) * C, (int64_t)V::D_OUT * C * 4, q, C);
    // a kind takes the accumulate flag at run time (one kernel for both)
    if (ACC || (V::RT && a.accum)) {
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
// With a.sw = 2 a workgroup holds the waves of two consecutive channel slabs of
// one (receiver, group): they share the staged A and A2 of each batch, the
// first wave forming A and the second A2.  A lone wave stages batches of
// kEdgeBatch3 edges, a pair batches of E3_FWD3_BATCH2.
constexpr int kEdgeBatch3 = 8;

template <class V, int G>
__device__ __forceinline__ void fwd3_task(const ConvArgs& a, int b, int sl, float* sA, float* sA2) {
  using F = typename V::template FG<G>;
  const int lane = threadIdx.x & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  int ch0, lanes;
  slab_of<1>(a.C, sl * a.sw + w, ch0, lanes);
  const bool act = lane < lanes;
  const int C = a.C, q = ch0 + lane;
  const int e0 = uniform(a.rowptr[b]), e1 = uniform(a.rowptr[b + 1]);
  float acc[F::NROW][1];
#pragma unroll
  for (int i = 0; i < F::NROW; ++i) acc[i][0] = 0.0f;
  for (int eb = e0; eb < e1; eb += a.fb) {
    const int n = imin(a.fb, e1 - eb);
    int my_e = 0, my_src = 0;
    if (lane < n) {
      my_e = a.eid[eb + lane];
      my_src = a.src[eb + lane];
      // a lone wave forms both pre-contractions; of a pair, wave w forms one
      for (int k = a.sw == 1 ? 0 : w; k < 2; k += a.sw) {
        const float* yk = k == 0 ? a.y : a.y2;
        float Y[V::D_SH];
#pragma unroll
        for (int i = 0; i < V::D_SH; ++i) Y[i] = yk[(int64_t)my_e * V::D_SH + i];
        F::make_A(Y, (k == 0 ? sA : sA2) + lane * F::NA);
      }
    }
    __syncthreads();
    if (act) {
      float xa[F::NXR][1], xda[F::NXR][1], sa[F::NPATH][1], sda[F::NPATH][1];
      float xb[F::NXR][1], xdb[F::NXR][1], sb[F::NPATH][1], sdb[F::NPATH][1];
      auto load = [&](int j, float (&xv)[F::NXR][1], float (&xdv)[F::NXR][1], float (&sv)[F::NPATH][1],
                      float (&sdv)[F::NPATH][1]) {
        const int64_t e = __builtin_amdgcn_readlane(my_e, j);
        const int64_t snd = __builtin_amdgcn_readlane(my_src, j);
        const RowBuf xr = row_buf(a.x + snd * x_rows<V>(a) * C, (int64_t)V::D_IN * C * 4, q, C);
        const RowBuf x2r = row_buf(a.x2 + snd * x_rows<V>(a) * C, (int64_t)V::D_IN * C * 4, q, C);
        const RowBuf sr = row_buf(a.s + e * p_rows<V>(a) * C, (int64_t)V::NP * C * 4, q, C);
        const RowBuf s2r = row_buf(a.s2 + e * p_rows<V>(a) * C, (int64_t)V::NP * C * 4, q, C);
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
    const RowBuf mb = row_buf(a.m + (int64_t)b * o_rows<V>(a) * C, (int64_t)V::D_OUT * C * 4, q, C);
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

// a.nslab counts slab groups of a.sw slabs here; blockDim.x = a.sw * kWave;
// dynamic LDS: fwd3_lds_bytes<V>(a)
template <class V>
__global__ __launch_bounds__(2 * kWave, E3_FWD_MIN_WAVES) void k_conv_fwd3(ConvArgs a) {
  extern __shared__ __align__(16) float lds3[];
  int b, g, sl;
  if (!task_of<V::NFG>(a, b, g, sl)) return;
  fwd3_dispatch<V, 0>(a, b, g, sl, lds3, lds3 + a.fb * V::MAX_NA_F);
}

template <class V>
size_t fwd3_lds_bytes(const ConvArgs& a) { return (size_t)2 * a.fb * V::MAX_NA_F * sizeof(float); }

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
    const RowBuf db = row_buf(a.dm + (int64_t)b * o_rows<V>(a) * C, (int64_t)V::D_OUT * C * 4, q, C);
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
      const RowBuf xb_ = row_buf(a.x + snd * x_rows<V>(a) * C, (int64_t)V::D_IN * C * 4, q, C);
#pragma unroll
      for (int i = 0; i < B::NXR; ++i) bld<CPL>(xb_, B::XROW[i], xv[i]);
    };
    auto load_s = [&](int j, float (&sv)[B::NPATH][CPL]) {
      if (!act) return;
      const int64_t e = __builtin_amdgcn_readlane(my_e, j);
      const RowBuf sb_ = row_buf(a.s + e * p_rows<V>(a) * C, (int64_t)V::NP * C * 4, q, C);
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
        const RowBuf dsb = row_buf(a.ds + e * p_rows<V>(a) * C, a.ds_row, q, C);
        // accumulating: the old ds of this edge is loaded before the contraction
        // starts, so that its latency is hidden behind the arithmetic (a kind
        // takes the flag at run time)
        constexpr bool MAYACC = ACC || V::RT;
        const bool acc_ds = ACC || (V::RT && a.accum);
        float old[MAYACC ? B::NPATH : 1][CPL];
        if constexpr (MAYACC) {
          if (acc_ds) {
#pragma unroll
            for (int i = 0; i < B::NPATH; ++i) bld<CPL>(dsb, B::PATH[i], old[i]);
          }
        }
        auto st = [&](int pl, const float (&v)[CPL]) {
          if constexpr (MAYACC) {
            if (acc_ds) {
              float o[CPL];
#pragma unroll
              for (int c = 0; c < CPL; ++c) o[c] = old[pl][c] + v[c];
              bst<CPL, kST>(dsb, B::PATH[pl], o);
              return;
            }
          }
          bst<CPL, kST>(dsb, B::PATH[pl], v);
        };
        float dyl[V::D_SH];
#pragma unroll
        for (int i = 0; i < V::D_SH; ++i) dyl[i] = 0.0f;
        B::template edge<E3_BWD_ALOAD_PIN != 0, CPL>(sA + j * B::NA, Yv, xv, sv, dmv, t, dyl, st);
#pragma unroll
        for (int i = 0; i < V::D_SH; ++i) dy[i] = dyl[i];
        {
          const RowBuf Tb = row_buf(a.T + slot * x_rows<V>(a) * C, a.t_row, q, C);
#pragma unroll
          for (int i = 0; i < B::NXR; ++i) bst<CPL, E3_T_STORE_AUX>(Tb, B::XROW[i], t[i]);
        }
      }
      const float tot = wave_reduce16(dy, lane);
      if ((lane & 3) == 0) a.DY[(dy_group<V, G>(a, eb + j) * a.nslab + sl) * 16 + (lane >> 2)] = tot;
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
    const RowBuf db = row_buf(a.dm + (int64_t)b * o_rows<V>(a) * C, (int64_t)V::D_OUT * C * 4, q, C);
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
      const RowBuf xr = row_buf(a.x + snd * x_rows<V>(a) * C, (int64_t)V::D_IN * C * 4, q, C);
      const RowBuf x2r = row_buf(a.x2 + snd * x_rows<V>(a) * C, (int64_t)V::D_IN * C * 4, q, C);
      const RowBuf sr = row_buf(a.s + e * p_rows<V>(a) * C, (int64_t)V::NP * C * 4, q, C);
      const RowBuf s2r = row_buf(a.s2 + e * p_rows<V>(a) * C, (int64_t)V::NP * C * 4, q, C);
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
        const RowBuf gsb = row_buf(a.ds + e * p_rows<V>(a) * C, (int64_t)V::NP * C * 4, q, C);
        auto st = [&](int pl, const float (&v)[1]) { bst<1, kST>(gsb, B::PATH[pl], v); };
        B::template edge3<1>(Yv, Y2v, xv, xdv, sv, sdv, dmv, t, dyl, st);
#pragma unroll
        for (int i = 0; i < V::D_SH; ++i) dy[i] = dyl[i];
        const RowBuf Tb = row_buf(a.T + slot * x_rows<V>(a) * C, (int64_t)V::D_IN * C * 4, q, C);
#pragma unroll
        for (int i = 0; i < B::NXR; ++i) bst<1, E3_T_STORE_AUX>(Tb, B::XROW[i], t[i]);
      }
      const float tot = wave_reduce16(dy, lane);
      if ((lane & 3) == 0) a.DY[(dy_group<V, G>(a, eb + j) * a.nslab + sl) * 16 + (lane >> 2)] = tot;
    };
#ifndef E3_BWD3_SINGLE
#define E3_BWD3_SINGLE 1
#endif
#if E3_BWD3_SINGLE
    for (int j = 0; j < n; ++j) {
      load(j, xa, xda, sa, sda);
      compute(j, xa, xda, sa, sda);
    }
    (void)xb, (void)xdb, (void)sb, (void)sdb;
#else
    load(0, xa, xda, sa, sda);
    for (int j = 0; j < n; j += 2) {
      if (j + 1 < n) load(j + 1, xb, xdb, sb, sdb);
      compute(j, xa, xda, sa, sda);
      if (j + 1 < n) {
        if (j + 2 < n) load(j + 2, xa, xda, sa, sda);
        compute(j + 1, xb, xdb, sb, sdb);
      }
    }
#endif
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

// Two waves per SIMD with each edge's rows loaded just before its contraction
// (E3_BWD3_SINGLE): 255 registers, no spill, 17.9 ms at the 24,000-atom box.
// Loading the next edge's rows during the contraction needs about 30 more
// registers: at two waves per SIMD it spilled 136 bytes per lane (26.6 ms), at
// one it ran 23.4 ms.
#ifndef E3_BWD3_MIN_WAVES
#define E3_BWD3_MIN_WAVES 2
#endif
template <class V>
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
  // float4 k of the lane at byte offset off + k * 64 * 16, all of it in the
  // lane offset (which the descriptor's range check covers): float4s past
  // D_in x C read as zero and are not stored
  E3_UNROLL(E3_DX_UNROLL)
  for (int t = s0; t < s1; ++t) {
    __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(T) + (int64_t)t * flat4 * 4, (short)0, (int)slot_bytes, 0x00020000);
#pragma unroll
    for (int k = 0; k < kDxVec; ++k)
      acc[k] += __builtin_bit_cast(f4v, __builtin_amdgcn_raw_buffer_load_b128(r, off + k * kWave * 16, 0, kNT));
  }
  if (accum) {  // old + this sum, so that accumulating equals adding a separate result
#pragma unroll
    for (int k = 0; k < kDxVec; ++k)
      acc[k] += __builtin_bit_cast(f4v, __builtin_amdgcn_raw_buffer_load_b128(o, off + k * kWave * 16, 0, 0));
  }
#pragma unroll
  for (int k = 0; k < kDxVec; ++k)
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u4v, acc[k]), o, off + k * kWave * 16, 0, kST);
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


// ------------------------------------------------------------ float64 builds
// The tensor product and the convolution in float64, the precision the paper
// measures its float32 kernels against (App. D, "Precision").  They run the
// same generated per-edge code (generic in the scalar type) in simpler
// skeletons than the float32 sweeps: one channel per lane, one 64-channel slab
// per wave, rows through 8-byte buffer loads, harmonic cotangents summed
// across the wave by a fixed butterfly.  Accuracy, not throughput, is their use.
struct RowBuf64 {
  __amdgpu_buffer_rsrc_t r;
  int voff;      // lane's channel, bytes
  int rowbytes;  // C * 8
};

__device__ __forceinline__ RowBuf64 row_buf64(const double* base, int64_t nbytes, int q, int C) {
  RowBuf64 b;
  b.r = __builtin_amdgcn_make_buffer_rsrc(const_cast<double*>(base), (short)0,
                                          (int)(nbytes < 0x7fffffff ? nbytes : 0x7fffffff), 0x00020000);
  b.voff = q * 8;
  b.rowbytes = C * 8;
  return b;
}

__device__ __forceinline__ void bld64(const RowBuf64& b, int row, double (&v)[1]) {
  typedef unsigned u2v __attribute__((ext_vector_type(2)));
  v[0] = __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(b.r, b.voff, row * b.rowbytes, 0));
  (void)sizeof(u2v);
}

__device__ __forceinline__ void bst64(const RowBuf64& b, int row, const double (&v)[1]) {
  typedef unsigned u2v __attribute__((ext_vector_type(2)));
  __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u2v, v[0]), b.r, b.voff, row * b.rowbytes, 0);
}

// Sum over the 64 lanes, the same fixed butterfly on every lane.
__device__ __forceinline__ double wave_sum64(double v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}

__device__ __forceinline__ void unit_of64(const double* __restrict__ vec, int64_t e, double& ux, double& uy,
                                          double& uz, double& inv) {
  const double vx = vec[3 * e], vy = vec[3 * e + 1], vz = vec[3 * e + 2];
  const double r2 = vx * vx + vy * vy + vz * vz;
  inv = r2 > 0.0 ? 1.0 / sqrt(r2) : 0.0;
  ux = vx * inv, uy = vy * inv, uz = vz * inv;
}

constexpr int kBatch64 = 8;  // rows / edges whose pre-contraction is staged per LDS batch

template <class V>
__global__ __launch_bounds__(kWave) void k_tp64(const double* __restrict__ x, const double* __restrict__ y,
                                                const double* __restrict__ w, double* __restrict__ z, int64_t rows,
                                                int C, int nslab, TpStr ts) {
  using F = typename V::TP;
  __shared__ __align__(32) double sA[kBatch64 * F::NA];
  const int lane = threadIdx.x;
  int sl;
  int64_t tile;
  if (!tile_of<false>(rows, kBatch64, nslab, tile, sl)) return;
  int ch0, lanes;
  slab_of<1>(C, sl, ch0, lanes);
  const int64_t r0 = tile * kBatch64;
  const int n = (int)((rows - r0) < kBatch64 ? (rows - r0) : kBatch64);
  if (lane < n) {
    double Y[V::D_SH];
#pragma unroll
    for (int i = 0; i < V::D_SH; ++i) Y[i] = y[(r0 + lane) * V::D_SH + i];
    F::make_A(Y, sA + lane * F::NA);
  }
  __syncthreads();
  if (lane >= lanes) return;
  const int q = ch0 + lane;
  for (int j = 0; j < n; ++j) {
    const int64_t r = r0 + j;
    double xv[F::NXR][1], wv[F::NPATH][1];
    const RowBuf64 xb = row_buf64(x + r * x_rows<V>(ts) * C, (int64_t)V::D_IN * C * 8, q, C);
    const RowBuf64 wb = row_buf64(w + r * p_rows<V>(ts) * C, (int64_t)V::NP * C * 8, q, C);
    const RowBuf64 zb = row_buf64(z + r * o_rows<V>(ts) * C, (int64_t)V::D_OUT * C * 8, q, C);
#pragma unroll
    for (int i = 0; i < F::NXR; ++i) bld64(xb, F::XROW[i], xv[i]);
#pragma unroll
    for (int i = 0; i < F::NPATH; ++i) bld64(wb, F::PATH[i], wv[i]);
    auto st = [&](int row, const double (&v)[1]) { bst64(zb, row, v); };
    F::template rows<1>(sA + j * F::NA, xv, wv, st);
  }
}

// Backward of one row group: dx, dw rows stored directly, dy summed over the
// wave's channels into a per-(row, group, slab) slot of DY.
struct Tpb64Args {
  const double* x;
  const double* y;
  const double* w;
  const double* dz;
  double* dx;
  double* dw;
  double* DY;  // [rows, NBG * nslab, 16]
  int64_t rows;
  int C;
  int nslab;
  int xr, pr, orr, ng, g0;  // a single-block kind inside a larger layout (as in ConvArgs)
};

template <class V, int G>
__device__ __forceinline__ void tpb64_task(const Tpb64Args& a, int64_t r0, int sl, double* sA, double* sY) {
  using B = typename V::template BG<G>;
  const int lane = threadIdx.x;
  int ch0, lanes;
  slab_of<1>(a.C, sl, ch0, lanes);
  const bool act = lane < lanes;
  const int C = a.C, q = ch0 + lane;
  const int n = (int)((a.rows - r0) < kBatch64 ? (a.rows - r0) : kBatch64);
  if (lane < n) {
    double Y[V::D_SH];
#pragma unroll
    for (int i = 0; i < V::D_SH; ++i) Y[i] = a.y[(r0 + lane) * V::D_SH + i];
#pragma unroll
    for (int i = 0; i < V::D_SH; ++i) sY[lane * V::D_SH + i] = Y[i];
    B::make_A(Y, sA + lane * B::NA);
  }
  __syncthreads();
  for (int j = 0; j < n; ++j) {
    const int64_t r = r0 + j;
    double dyl[V::D_SH];
#pragma unroll
    for (int i = 0; i < V::D_SH; ++i) dyl[i] = 0.0;
    if (act) {
      const RowBuf64 xb = row_buf64(a.x + r * x_rows<V>(a) * C, (int64_t)V::D_IN * C * 8, q, C);
      const RowBuf64 wb = row_buf64(a.w + r * p_rows<V>(a) * C, (int64_t)V::NP * C * 8, q, C);
      const RowBuf64 zb = row_buf64(a.dz + r * o_rows<V>(a) * C, (int64_t)V::D_OUT * C * 8, q, C);
      double xv[B::NXR][1], wv[B::NPATH][1], dzv[B::NROW][1], t[B::NXR][1], Yv[V::D_SH];
#pragma unroll
      for (int i = 0; i < B::NXR; ++i) bld64(xb, B::XROW[i], xv[i]), t[i][0] = 0.0;
#pragma unroll
      for (int i = 0; i < B::NPATH; ++i) bld64(wb, B::PATH[i], wv[i]);
#pragma unroll
      for (int i = 0; i < B::NROW; ++i) bld64(zb, B::OROW[i], dzv[i]);
#pragma unroll
      for (int i = 0; i < V::D_SH; ++i) Yv[i] = sY[j * V::D_SH + i];
      const RowBuf64 dwb = row_buf64(a.dw + r * p_rows<V>(a) * C, (int64_t)V::NP * C * 8, q, C);
      auto st = [&](int pl, const double (&v)[1]) { bst64(dwb, B::PATH[pl], v); };
      B::template edge<false, 1>(sA + j * B::NA, Yv, xv, wv, dzv, t, dyl, st);
      const RowBuf64 dxb = row_buf64(a.dx + r * x_rows<V>(a) * C, (int64_t)V::D_IN * C * 8, q, C);
#pragma unroll
      for (int i = 0; i < B::NXR; ++i) bst64(dxb, B::XROW[i], t[i]);
    }
#pragma unroll
    for (int i = 0; i < V::D_SH; ++i) {
      const double tot = wave_sum64(dyl[i]);
      if (lane == 0) a.DY[(dy_group<V, G>(a, r) * a.nslab + sl) * 16 + i] = tot;
    }
  }
}

template <class V, int G>
__device__ __forceinline__ void tpb64_dispatch(const Tpb64Args& a, int64_t r0, int g, int sl, double* sA,
                                               double* sY) {
  if constexpr (G < V::NBG) {
    if (g == G)
      tpb64_task<V, G>(a, r0, sl, sA, sY);
    else
      tpb64_dispatch<V, G + 1>(a, r0, g, sl, sA, sY);
  }
}

template <class V>
__global__ __launch_bounds__(kWave, 1) void k_tp_bwd64(Tpb64Args a) {
  __shared__ __align__(32) double smem[kBatch64 * (V::MAX_NA_B + V::D_SH)];
  int t;
  int64_t tile;
  if (!tile_of<false>(a.rows, kBatch64, V::NBG * a.nslab, tile, t)) return;
  tpb64_dispatch<V, 0>(a, tile * kBatch64, t / a.nslab, t % a.nslab, smem, smem + kBatch64 * V::MAX_NA_B);
}

// dy of each row (or live edge): the sum of its per-(group, slab) partials, in order.
template <class V>
__global__ __launch_bounds__(256) void k_dy_sum64(const double* __restrict__ DY, const int* __restrict__ eid,
                                                  double* __restrict__ dy, int64_t n, int nslab) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t r = i / V::D_SH;
  const int c = (int)(i % V::D_SH);
  if (r >= n) return;
  double v = 0.0;
  for (int g = 0; g < V::NBG * nslab; ++g) v += DY[(r * V::NBG * nslab + g) * 16 + c];
  dy[(eid ? (int64_t)eid[r] : r) * V::D_SH + c] = v;
}

// Convolution forward: one wave per (receiver, forward group, slab); the
// receiver's sums in registers, stored once.
template <class V, int G>
__device__ __forceinline__ void fwd64_task(const ConvArgs& a, const double* x, const double* vec, const double* s,
                                           double* m, int b, int sl, double* sA) {
  using F = typename V::template FG<G>;
  const int lane = threadIdx.x;
  int ch0, lanes;
  slab_of<1>(a.C, sl, ch0, lanes);
  const bool act = lane < lanes;
  const int C = a.C, q = ch0 + lane;
  const int e0 = uniform(a.rowptr[b]), e1 = uniform(a.rowptr[b + 1]);
  double acc[F::NROW][1];
#pragma unroll
  for (int i = 0; i < F::NROW; ++i) acc[i][0] = 0.0;
  for (int eb = e0; eb < e1; eb += kBatch64) {
    const int n = imin(kBatch64, e1 - eb);
    int my_e = 0, my_src = 0;
    if (lane < n) {
      my_e = a.eid[eb + lane];
      my_src = a.src[eb + lane];
      double ux, uy, uz, inv, Y[V::D_SH];
      unit_of64(vec, my_e, ux, uy, uz, inv);
      V::sh(ux, uy, uz, Y);
      F::make_A(Y, sA + lane * F::NA);
    }
    __syncthreads();
    if (act) {
      for (int j = 0; j < n; ++j) {
        const int64_t e = __builtin_amdgcn_readlane(my_e, j);
        const int64_t snd = __builtin_amdgcn_readlane(my_src, j);
        const RowBuf64 xb = row_buf64(x + snd * x_rows<V>(a) * C, (int64_t)V::D_IN * C * 8, q, C);
        const RowBuf64 sb = row_buf64(s + e * p_rows<V>(a) * C, (int64_t)V::NP * C * 8, q, C);
        double xv[F::NXR][1], sv[F::NPATH][1];
#pragma unroll
        for (int i = 0; i < F::NXR; ++i) bld64(xb, F::XROW[i], xv[i]);
#pragma unroll
        for (int i = 0; i < F::NPATH; ++i) bld64(sb, F::PATH[i], sv[i]);
        F::template edge<1>(sA + j * F::NA, xv, sv, acc);
      }
    }
    __syncthreads();
  }
  if (act) {
    const RowBuf64 mb = row_buf64(m + (int64_t)b * o_rows<V>(a) * C, (int64_t)V::D_OUT * C * 8, q, C);
#pragma unroll
    for (int i = 0; i < F::NROW; ++i) bst64(mb, F::OROW[i], acc[i]);
  }
}

template <class V, int G>
__device__ __forceinline__ void fwd64_dispatch(const ConvArgs& a, const double* x, const double* vec,
                                               const double* s, double* m, int b, int g, int sl, double* sA) {
  if constexpr (G < V::NFG) {
    if (g == G)
      fwd64_task<V, G>(a, x, vec, s, m, b, sl, sA);
    else
      fwd64_dispatch<V, G + 1>(a, x, vec, s, m, b, g, sl, sA);
  }
}

template <class V>
__global__ __launch_bounds__(kWave, 1) void k_conv_fwd64(ConvArgs a, const double* __restrict__ x,
                                                         const double* __restrict__ vec,
                                                         const double* __restrict__ s, double* __restrict__ m) {
  __shared__ __align__(32) double sA[kBatch64 * V::MAX_NA_F];
  int b, g, sl;
  if (!task_of<V::NFG>(a, b, g, sl)) return;
  fwd64_dispatch<V, 0>(a, x, vec, s, m, b, g, sl, sA);
}

// Convolution backward sweep in receiver order: ds per edge, the x-cotangent
// partials T at the edge's sender-CSR slot, the per-wave harmonic cotangents.
struct Conv64Out {
  const double* x;
  const double* vec;
  const double* s;
  const double* dm;
  double* ds;
  double* T;   // [n_live, D_in, C]
  double* DY;  // [n_live, NBG * nslab, 16]
};

template <class V, int G>
__device__ __forceinline__ void bwd64_task(const ConvArgs& a, const Conv64Out& o, int b, int sl, double* sA,
                                           double* sY) {
  using B = typename V::template BG<G>;
  const int lane = threadIdx.x;
  int ch0, lanes;
  slab_of<1>(a.C, sl, ch0, lanes);
  const bool act = lane < lanes;
  const int C = a.C, q = ch0 + lane;
  const int e0 = uniform(a.rowptr[b]), e1 = uniform(a.rowptr[b + 1]);
  if (e0 == e1) return;
  double dmv[B::NROW][1];
  if (act) {
    const RowBuf64 db = row_buf64(o.dm + (int64_t)b * o_rows<V>(a) * C, (int64_t)V::D_OUT * C * 8, q, C);
#pragma unroll
    for (int i = 0; i < B::NROW; ++i) bld64(db, B::OROW[i], dmv[i]);
  }
  for (int eb = e0; eb < e1; eb += kBatch64) {
    const int n = imin(kBatch64, e1 - eb);
    int my_e = 0, my_src = 0, my_slot = 0;
    if (lane < n) {
      my_e = a.eid[eb + lane];
      my_src = a.src[eb + lane];
      my_slot = a.r2s[eb + lane];
      double ux, uy, uz, inv, Y[V::D_SH];
      unit_of64(o.vec, my_e, ux, uy, uz, inv);
      V::sh(ux, uy, uz, Y);
#pragma unroll
      for (int i = 0; i < V::D_SH; ++i) sY[lane * V::D_SH + i] = Y[i];
      B::make_A(Y, sA + lane * B::NA);
    }
    __syncthreads();
    for (int j = 0; j < n; ++j) {
      const int64_t e = __builtin_amdgcn_readlane(my_e, j);
      const int64_t snd = __builtin_amdgcn_readlane(my_src, j);
      const int64_t slot = __builtin_amdgcn_readlane(my_slot, j);
      double dyl[V::D_SH];
#pragma unroll
      for (int i = 0; i < V::D_SH; ++i) dyl[i] = 0.0;
      if (act) {
        const RowBuf64 xb = row_buf64(o.x + snd * x_rows<V>(a) * C, (int64_t)V::D_IN * C * 8, q, C);
        const RowBuf64 sb = row_buf64(o.s + e * p_rows<V>(a) * C, (int64_t)V::NP * C * 8, q, C);
        double xv[B::NXR][1], sv[B::NPATH][1], t[B::NXR][1], Yv[V::D_SH];
#pragma unroll
        for (int i = 0; i < B::NXR; ++i) bld64(xb, B::XROW[i], xv[i]), t[i][0] = 0.0;
#pragma unroll
        for (int i = 0; i < B::NPATH; ++i) bld64(sb, B::PATH[i], sv[i]);
#pragma unroll
        for (int i = 0; i < V::D_SH; ++i) Yv[i] = sY[j * V::D_SH + i];
        const RowBuf64 dsb = row_buf64(o.ds + e * p_rows<V>(a) * C, (int64_t)V::NP * C * 8, q, C);
        auto st = [&](int pl, const double (&v)[1]) { bst64(dsb, B::PATH[pl], v); };
        B::template edge<false, 1>(sA + j * B::NA, Yv, xv, sv, dmv, t, dyl, st);
        const RowBuf64 Tb = row_buf64(o.T + slot * x_rows<V>(a) * C, (int64_t)V::D_IN * C * 8, q, C);
#pragma unroll
        for (int i = 0; i < B::NXR; ++i) bst64(Tb, B::XROW[i], t[i]);
      }
#pragma unroll
      for (int i = 0; i < V::D_SH; ++i) {
        const double tot = wave_sum64(dyl[i]);
        if (lane == 0) o.DY[(dy_group<V, G>(a, eb + j) * a.nslab + sl) * 16 + i] = tot;
      }
    }
    __syncthreads();
  }
}

template <class V, int G>
__device__ __forceinline__ void bwd64_dispatch(const ConvArgs& a, const Conv64Out& o, int b, int g, int sl,
                                               double* sA, double* sY) {
  if constexpr (G < V::NBG) {
    if (g == G)
      bwd64_task<V, G>(a, o, b, sl, sA, sY);
    else
      bwd64_dispatch<V, G + 1>(a, o, b, g, sl, sA, sY);
  }
}

template <class V>
__global__ __launch_bounds__(kWave, 1) void k_conv_bwd64(ConvArgs a, Conv64Out o) {
  __shared__ __align__(32) double smem[kBatch64 * (V::MAX_NA_B + V::D_SH)];
  int b, g, sl;
  if (!task_of<V::NBG>(a, b, g, sl)) return;
  bwd64_dispatch<V, 0>(a, o, b, g, sl, smem, smem + kBatch64 * V::MAX_NA_B);
}

// dx[node] = sum of its partial rows in sender-CSR order (one wave per node
// and 64-channel slab, rows walked in registers).
__global__ __launch_bounds__(kWave) void k_conv_bwd_dx64(const double* __restrict__ T, double* __restrict__ dx,
                                                         const int* __restrict__ rowptr_s, int n_nodes, int D_in,
                                                         int C, int nslab) {
  const int64_t bid = blockIdx.x;
  const int node = (int)(bid / nslab), sl = (int)(bid % nslab);
  if (node >= n_nodes) return;
  const int q = sl * kWave + threadIdx.x;
  if (q >= C) return;
  const int s0 = uniform(rowptr_s[node]), s1 = uniform(rowptr_s[node + 1]);
  for (int i = 0; i < D_in; ++i) {
    double acc = 0.0;
    for (int t = s0; t < s1; ++t) acc += T[((int64_t)t * D_in + i) * C + q];
    dx[((int64_t)node * D_in + i) * C + q] = acc;
  }
}

// dvec of each live edge from its harmonic cotangent (summed over groups).
template <class V>
__global__ __launch_bounds__(256) void k_conv_bwd_dvec64(const double* __restrict__ vec,
                                                         const double* __restrict__ DY, const int* __restrict__ eid,
                                                         double* __restrict__ dvec, int64_t n_live, int nslab) {
  const int64_t pos = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (pos >= n_live) return;
  const int64_t e = eid[pos];
  double dY[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) dY[i] = 0.0;
  for (int g = 0; g < V::NBG * nslab; ++g)
#pragma unroll
    for (int i = 0; i < V::D_SH; ++i) dY[i] += DY[(pos * V::NBG * nslab + g) * 16 + i];
  double ux, uy, uz, inv, gx, gy, gz;
  unit_of64(vec, e, ux, uy, uz, inv);
  V::sh_grad(ux, uy, uz, dY, gx, gy, gz);
  const double ug = ux * gx + uy * gy + uz * gz;
  dvec[3 * e] = (gx - ux * ug) * inv;
  dvec[3 * e + 1] = (gy - uy * ug) * inv;
  dvec[3 * e + 2] = (gz - uz * ug) * inv;
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
__device__ __forceinline__ void radial_quad(const RowBuf& wb, int wrows, const float* sH, int q4, int K,
                                            const int (&path)[NPATH], f4v (&s4)[NPATH]) {
  const int lane = threadIdx.x;
#pragma unroll
  for (int p = 0; p < NPATH; ++p) s4[p] = f4v{0.0f, 0.0f, 0.0f, 0.0f};
  for (int j = 0; j < K; ++j) {
    const float hv = sH[(q4 + (lane & 3)) * kRadKMax + j];
    float wv[NPATH][1];
#pragma unroll
    for (int p = 0; p < NPATH; ++p) bld<1>(wb, j * wrows + path[p], wv[p]);
#pragma unroll
    for (int p = 0; p < NPATH; ++p) s4[p] = __builtin_amdgcn_mfma_f32_4x4x1f32(hv, wv[p][0], s4[p], 0, 0, 0);
  }
}

// Bytes of W [K, P, C] a kernel may read from its base: all of it for a
// compiled layout; for a single-block kind (base at its first path, row
// stride P) the K row sets up to its own last path.
template <class V>
__device__ __forceinline__ int64_t w_bytes(const ConvArgs& a) {
  if constexpr (V::RT) return ((int64_t)(a.K - 1) * a.pr + V::NP) * a.C * 4;
  else return (int64_t)a.K * V::NP * a.C * 4;
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
  const RowBuf wb = row_buf(a.W, w_bytes<V>(a), q, C);
  float wr[KR > 0 ? KR : 1][F::NPATH];
  if constexpr (KR > 0) {
#pragma unroll
    for (int j = 0; j < KR; ++j)
#pragma unroll
      for (int p = 0; p < F::NPATH; ++p) {
        float v[1] = {0.0f};
        if (j < a.K) bld<1>(wb, j * p_rows<V>(a) + F::PATH[p], v);
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
      const RowBuf xr = row_buf(a.x + snd * x_rows<V>(a) * C, (int64_t)V::D_IN * C * 4, q, C);
#pragma unroll
      for (int i = 0; i < F::NXR; ++i) bld<1>(xr, F::XROW[i], xv[i]);
    };
    load_x(0, xa);
    for (int q4 = 0; q4 < n; q4 += 4) {
      f4v s4[F::NPATH];
      if constexpr (KR > 0)
        radial_quad_reg<V, F::NPATH, (KR > 0 ? KR : 1)>(wr, sH, q4, s4);
      else
        radial_quad<V, F::NPATH>(wb, p_rows<V>(a), sH, q4, a.K, F::PATH, s4);
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
    const RowBuf mb = row_buf(a.m + (int64_t)b * o_rows<V>(a) * C, (int64_t)V::D_OUT * C * 4, q, C);
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
    const RowBuf db = row_buf(a.dm + (int64_t)b * o_rows<V>(a) * C, (int64_t)V::D_OUT * C * 4, q, C);
#pragma unroll
    for (int i = 0; i < B::NROW; ++i) bld<1>(db, B::OROW[i], dmv[i]);
  }
  const RowBuf wb = row_buf(a.W, w_bytes<V>(a), q, C);
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
      const RowBuf xr = row_buf(a.x + snd * x_rows<V>(a) * C, (int64_t)V::D_IN * C * 4, q, C);
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
        const RowBuf dsb = row_buf(a.ds + e * p_rows<V>(a) * C, (int64_t)V::NP * C * 4, q, C);
        auto st = [&](int pl, const float (&v)[1]) { bst<1, kST>(dsb, B::PATH[pl], v); };
        float dyl[V::D_SH];
#pragma unroll
        for (int i = 0; i < V::D_SH; ++i) dyl[i] = 0.0f;
        B::template edge<false, 1>(sA + j * B::NA, Yv, xv, sv, dmv, t, dyl, st);
#pragma unroll
        for (int i = 0; i < V::D_SH; ++i) dy[i] = dyl[i];
        const RowBuf Tb = row_buf(a.T + slot * x_rows<V>(a) * C, (int64_t)V::D_IN * C * 4, q, C);
#pragma unroll
        for (int i = 0; i < B::NXR; ++i) bst<1, E3_T_STORE_AUX>(Tb, B::XROW[i], t[i]);
      }
      const float tot = wave_reduce16(dy, lane);
      if ((lane & 3) == 0) a.DY[(dy_group<V, G>(a, eb + j) * a.nslab + sl) * 16 + (lane >> 2)] = tot;
    };
    load_x(0, xa);
    for (int q4 = 0; q4 < n; q4 += 4) {
      f4v s4[B::NPATH];
      radial_quad<V, B::NPATH>(wb, p_rows<V>(a), sH, q4, a.K, B::PATH, s4);
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
// lane l owning float4 columns (kGradF sl + f) 64 + l (f < kGradF).  The dW outer products
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
#ifndef E3_GRAD_F
#define E3_GRAD_F 2
#endif
#ifndef E3_GRAD_WAVES
#define E3_GRAD_WAVES 8192
#endif
// float4 columns per lane: E3_GRAD_F for K <= 8; one for K <= 16, whose
// accumulators would otherwise leave one wave per SIMD
constexpr int grad_f(int KQ) { return KQ == 2 ? E3_GRAD_F : 1; }
constexpr int kGradRows = E3_GRAD_ROWS;  // rows whose loads are issued together

template <int KQ>
__global__ __launch_bounds__(kWave) void k_rad_grad(const float* __restrict__ DS, const float* __restrict__ h,
                                                    const float* __restrict__ W, float* __restrict__ dWp,
                                                    float* __restrict__ DHp, int64_t n_rows, int PC4, int K,
                                                    int nsl4, int rows_per) {
  static_assert(KQ == 2 || KQ == 4, "K <= 8 or K <= 16");
  constexpr int NV = 4 * KQ;
  constexpr int kGradF = grad_f(KQ);
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
// A block takes 64 consecutive entries; its kDwSplit waves each add every
// kDwSplit-th chunk (in chunk order) and the first wave adds their sums in
// wave order, so the order of every addition is fixed.
constexpr int kDwSplit = 8;

__global__ __launch_bounds__(kWave* kDwSplit) void k_rad_dw_sum(const float* __restrict__ dWp,
                                                                float* __restrict__ dW, int64_t n, int nchunk) {
  __shared__ float part[kDwSplit][kWave];
  const int o = threadIdx.x % kWave, g = threadIdx.x / kWave;
  const int64_t i = (int64_t)blockIdx.x * kWave + o;
  float s = 0.0f;
  if (i < n)
    for (int c = g; c < nchunk; c += kDwSplit) s += dWp[(int64_t)c * n + i];
  part[g][o] = s;
  __syncthreads();
  if (g == 0 && i < n) {
    float t = part[0][o];
#pragma unroll
    for (int k = 1; k < kDwSplit; ++k) t += part[k][o];
    dW[i] = t;
  }
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


unsigned blocks_for(int64_t n, int t) { return (unsigned)std::max<int64_t>(1, (n + t - 1) / t); }

}  // namespace

// ============================================================ handles
struct RecPlan;  // device tables of the record path (convr.hip)

struct e3_plan {
  e3b::Layout lay;
  std::vector<e3b::Record> recs;
  int variant = -1;
  // Channels per lane of the forward / tensor-product / dx kernels (the
  // backward sweep always uses 1) and the number of 64-lane channel slabs.
  int cpl_f = 0, cpl_b = 0, nslab_f = 0, nslab_b = 0;
  // A layout without a compiled variant runs on the record path, whose
  // tables are uploaded at plan creation (null when that was not possible).
  RecPlan* rec = nullptr;
  std::string no_rec_reason;  // why not, when rec is null
  // The composed path (a layout without a compiled variant, every x block of
  // degree <= 3): per x block with paths, its kind and offsets; the x rows of
  // blocks without paths (their cotangent rows are zero); the harmonic-partial
  // groups over all blocks.
  struct KindBlock {
    int kind, x_off, k0, o_off, g0;
  };
  bool composed = false;
  std::vector<KindBlock> kblocks;
  std::vector<std::pair<int, int>> pathless;  // (first x row, rows)
  int kng = 0;
  e3_plan() = default;
  e3_plan(const e3_plan&) = delete;
  e3_plan& operator=(const e3_plan&) = delete;
  ~e3_plan();
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

struct Ws {
  size_t t_bytes, dy_bytes;
};

// Scratch of the radial backward: T and DY as in the plain backward, then ds
// by edge id (all E rows when any edge is live), the dW partials of each row
// chunk and the dh partials of each column slab.
struct RadWs {
  size_t t, dy, ds, dwp, dhp;
  int nchunk, rows_per, nsl4, nv, pc4;
  size_t total() const { return t + dy + ds + dwp + dhp; }
};

// ---- layouts without a compiled variant (convr.hip): the composed path
// (single-block kinds run block by block) or, when forced or when no kind
// fits, the record path (the plan's coupling records walked at run time).
// rec_fwd / rec_bwd take the receiver graph g, or g == null for the tensor
// product over `rows` rows (s is w, m is z, ds is dw, dx written directly,
// with no workspace share for it); they run whichever of the two the plan has.
e3_status comp_create(e3_plan* p);         // matches every x block with a kind
e3_status rec_create(e3_plan* p);          // builds and uploads the tables
bool rec_ready(const e3_plan* p);          // tables on a device
e3_status rec_check(const e3_plan* p);     // ready, and their device is current
Ws rec_ws(const e3_plan* p, const e3_graph* g);
size_t rec_tp_ws(const e3_plan* p, int64_t rows);
e3_status rec_fwd(const e3_plan* p, const e3_graph* g, int64_t rows, const float* x, const float* vec,
                  const float* y, const float* s, float* m, int accum, hipStream_t st);
e3_status rec_bwd(const e3_plan* p, const e3_graph* g, int64_t rows, const float* x, const float* vec,
                  const float* y, const float* s, const float* dm, float* dx, float* dvec, float* dy, float* ds,
                  int accum, void* ws, hipStream_t st);
// the composed path's double backward (fused sweeps per block)
e3_status comp_bwd2(const e3_plan* p, const e3_graph* g, const float* x, const float* y, const float* s,
                    const float* dm, const float* ddx, const float* ddy, const float* dds, float* gx, float* gy,
                    float* gs, float* gdm, void* ws, hipStream_t st);
// the composed path's fused radial weights
RadWs comp_rad_ws(const e3_plan* p, const e3_graph* g, int K);
e3_status comp_fwd_rad(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* h,
                       const float* W, int K, float* m, hipStream_t st);
e3_status comp_bwd_rad(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* h,
                       const float* W, int K, const float* dm, float* dx, float* dvec, float* dh, float* dW,
                       void* ws, hipStream_t st);
// the composed path's float64 builds
Ws comp_ws64(const e3_plan* p, const e3_graph* g);
size_t comp_tp_ws64(const e3_plan* p, int64_t rows);
e3_status comp_fwd64(const e3_plan* p, const e3_graph* g, const double* x, const double* vec, const double* s,
                     double* m, hipStream_t st);
e3_status comp_bwd64(const e3_plan* p, const e3_graph* g, const double* x, const double* vec, const double* s,
                     const double* dm, double* dx, double* dvec, double* ds, void* ws, hipStream_t st);
e3_status comp_tp64(const e3_plan* p, const double* x, const double* y, const double* w, double* z, int64_t rows,
                    hipStream_t st);
e3_status comp_tpb64(const e3_plan* p, const double* x, const double* y, const double* w, const double* dz,
                     double* dx, double* dy, double* dw, void* ws, int64_t rows, hipStream_t st);


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
  // float64 builds
  e3_status (*tp64)(const e3_plan*, const double*, const double*, const double*, double*, int64_t, hipStream_t);
  e3_status (*tpb64)(const e3_plan*, const double*, const double*, const double*, const double*, double*, double*,
                     double*, void*, int64_t, hipStream_t);
  size_t (*tpws64)(const e3_plan*, int64_t);
  e3_status (*fwd64)(const e3_plan*, const e3_graph*, const double*, const double*, const double*, double*,
                     hipStream_t);
  e3_status (*bwd64)(const e3_plan*, const e3_graph*, const double*, const double*, const double*, const double*,
                     double*, double*, double*, void*, hipStream_t);
  Ws (*ws64)(const e3_plan*, const e3_graph*);
};

// ---- single-block kinds: the generated code of one x block (degree <= 3,
// all its paths or its natural-parity ones) under given harmonics and output
// degrees, run with the strides and offsets of a larger layout, block by
// block, for layouts without a compiled variant (the composed path).
struct KindCall {
  int xr, pr, orr;  // rows of the whole layout: x / dx per node, s / ds per edge, m / dm per node
  int ng, g0;       // harmonic-partial groups of the whole layout, and this block's first
};

struct KindOps {
  const char* sig;
  int d_in, d_sh, d_out, np, lsh, nbg;
  // the forward sweep of the block's output rows (x, s, m offset to the block)
  e3_status (*fwd)(const e3_plan*, const e3_graph*, const float* x, const float* vec, const float* y,
                   const float* s, float* m, int accum, const KindCall&, hipStream_t);
  // the backward edge sweep of the block: its ds rows, its rows of the
  // x-cotangent partials T, its harmonic partial groups
  e3_status (*bwd)(const e3_plan*, const e3_graph*, const float* x, const float* vec, const float* y,
                   const float* s, const float* dm, float* T, int64_t t_row, float* DY, float* ds, int64_t ds_row,
                   int accum_ds, const KindCall&, hipStream_t);
  e3_status (*tp)(const e3_plan*, const float* x, const float* y, const float* w, float* z, int64_t rows,
                  const KindCall&, hipStream_t);
  e3_status (*tpb)(const e3_plan*, const float* x, const float* y, const float* w, const float* dz, float* dx,
                   float* dw, float* DY, int64_t rows, const KindCall&, hipStream_t);
  // float64 builds (one channel per lane)
  e3_status (*fwd64)(const e3_plan*, const e3_graph*, const double* x, const double* vec, const double* s,
                     double* m, const KindCall&, hipStream_t);
  e3_status (*bwd64)(const e3_plan*, const e3_graph*, const double* x, const double* vec, const double* s,
                     const double* dm, double* T, double* DY, double* ds, const KindCall&, hipStream_t);
  e3_status (*tp64)(const e3_plan*, const double* x, const double* y, const double* w, double* z, int64_t rows,
                    const KindCall&, hipStream_t);
  e3_status (*tpb64)(const e3_plan*, const double* x, const double* y, const double* w, const double* dz,
                     double* dx, double* dw, double* DY, int64_t rows, const KindCall&, hipStream_t);
  // fused radial weights: W offset to the block's first path, row stride P
  e3_status (*rfwd)(const e3_plan*, const e3_graph*, const float* x, const float* vec, const float* h,
                    const float* W, int K, float* m, const KindCall&, hipStream_t);
  e3_status (*rbwd)(const e3_plan*, const e3_graph*, const float* x, const float* vec, const float* h,
                    const float* W, int K, const float* dm, float* T, float* DY, float* DS, const KindCall&,
                    hipStream_t);
  // the double backward's three forward terms and three backward terms, each in one sweep
  e3_status (*fwd3)(const e3_plan*, const e3_graph*, const float* x, const float* x2, const float* y,
                    const float* y2, const float* s, const float* s2, float* m, const KindCall&, hipStream_t);
  e3_status (*bwd3)(const e3_plan*, const e3_graph*, const float* x, const float* x2, const float* y,
                    const float* y2, const float* s, const float* s2, const float* dm, float* T, float* DY,
                    float* gs, const KindCall&, hipStream_t);
};

namespace {

size_t align256(size_t n) { return (n + 255) & ~size_t(255); }


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

// Slabs of the three-term forward: one channel per lane; the waves of two
// consecutive slabs share a workgroup when there are two or more slabs (an odd
// last slab's partner wave only forms A2).
inline void fwd3_slabs(ConvArgs& a) {
  const int nslab = (a.C + kWave - 1) / kWave;
  a.sw = E3_FWD3_PAIR && nslab >= 2 ? 2 : 1;
  a.nslab = (nslab + a.sw - 1) / a.sw;
  a.fb = a.sw == 2 ? E3_FWD3_BATCH2 : kEdgeBatch3;
}

// The double backward's three forward terms in one launch (k_conv_fwd3):
// m = conv(x2, y, s) + conv(x, y2, s) + conv(x, y, s2), overwritten.
template <class V>
e3_status run_fwd3(const e3_plan* p, const e3_graph* g, const float* x, const float* x2, const float* y,
                   const float* y2, const float* s, const float* s2, float* m, hipStream_t st) {
  ConvArgs a = base_args(p, g);
  a.x = x, a.x2 = x2, a.y = y, a.y2 = y2, a.s = s, a.s2 = s2, a.m = m;
  fwd3_slabs(a);
  if (g->n_nodes == 0) return E3_OK;
  const unsigned grid = (unsigned)(kXcd * a.chunk * V::NFG * a.nslab);
  {
    TimedLaunch t_("conv_fwd3", st);
    hipLaunchKernelGGL((k_conv_fwd3<V>), dim3(grid), dim3(a.sw * kWave), fwd3_lds_bytes<V>(a), st, a);
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
    hipLaunchKernelGGL((k_tp<V, CPL>), grid, dim3(kWave), 0, st, x, y, w, z, rows, p->lay.C, p->nslab_f, TpStr{});
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


// np: paths of the layout; b: the plain backward's scratch.
inline RadWs rad_ws_of(const e3_plan* p, const e3_graph* g, int K, int np, Ws b) {
  RadWs w{};
  w.t = b.t_bytes, w.dy = b.dy_bytes;
  const int64_t pc = (int64_t)np * p->lay.C, nl = g->n_live > 0 ? g->n_edges : 0;
  w.pc4 = (int)(pc / 4);
  const int f = grad_f(K <= 8 ? 2 : 4);
  w.nsl4 = (w.pc4 + kWave * f - 1) / (kWave * f);
  w.nv = K <= 8 ? 8 : 16;
  // about E3_GRAD_WAVES waves in the gradient kernel, at least 256 rows each
  const int64_t want = std::max<int64_t>(1, E3_GRAD_WAVES / w.nsl4);
  const int64_t nch = std::min<int64_t>(want, std::max<int64_t>(1, (nl + 255) / 256));
  w.rows_per = (int)std::max<int64_t>(1, (nl + nch - 1) / nch);
  w.nchunk = (int)((nl + w.rows_per - 1) / w.rows_per);
  w.ds = align256((size_t)nl * pc * sizeof(float));
  w.dwp = align256((size_t)w.nchunk * K * pc * sizeof(float));
  w.dhp = align256((size_t)nl * w.nsl4 * w.nv * sizeof(float));
  return w;
}

template <class V>
RadWs rad_ws(const e3_plan* p, const e3_graph* g, int K) {
  return rad_ws_of(p, g, K, V::NP, bwd_ws<V>(p, g));
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
    hipLaunchKernelGGL(k_rad_dw_sum, dim3(blocks_for(n, kWave)), dim3(kWave * kDwSplit), 0, st, dWp, dW, n,
                       w.nchunk);
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




// ---- float64 builds (one channel per lane)
inline int nslab64(const e3_plan* p) { return (p->lay.C + kWave - 1) / kWave; }

template <class V>
Ws bwd_ws64(const e3_plan* p, const e3_graph* g) {
  Ws w;
  w.t_bytes = align256((size_t)g->n_live * V::D_IN * p->lay.C * sizeof(double));
  w.dy_bytes = align256((size_t)g->n_live * V::NBG * nslab64(p) * 16 * sizeof(double));
  return w;
}

template <class V>
size_t tp_ws64(const e3_plan* p, int64_t rows) {
  return align256((size_t)rows * V::NBG * nslab64(p) * 16 * sizeof(double));
}

template <class V>
e3_status run_tp64(const e3_plan* p, const double* x, const double* y, const double* w, double* z, int64_t rows,
                   hipStream_t st) {
  const int nsl = nslab64(p);
  const int64_t grid = tile_grid(false, rows, kBatch64, nsl);
  if (grid > 0x7fffffff) return E3_ERR_INVALID_ARG;
  TimedLaunch t_("tp_fwd_f64", st);
  hipLaunchKernelGGL((k_tp64<V>), dim3((unsigned)grid), dim3(kWave), 0, st, x, y, w, z, rows, p->lay.C, nsl,
                     TpStr{});
  E3_HIP(hipGetLastError());
  return E3_OK;
}

template <class V>
e3_status run_tp_bwd64(const e3_plan* p, const double* x, const double* y, const double* w, const double* dz,
                       double* dx, double* dy, double* dw, void* ws, int64_t rows, hipStream_t st) {
  const int nsl = nslab64(p);
  Tpb64Args a{x, y, w, dz, dx, dw, reinterpret_cast<double*>(ws), rows, p->lay.C, nsl};
  const int64_t grid = tile_grid(false, rows, kBatch64, V::NBG * nsl);
  if (grid > 0x7fffffff) return E3_ERR_INVALID_ARG;
  {
    TimedLaunch t_("tp_bwd_f64", st);
    hipLaunchKernelGGL((k_tp_bwd64<V>), dim3((unsigned)grid), dim3(kWave), 0, st, a);
    E3_HIP(hipGetLastError());
  }
  TimedLaunch t_("tp_bwd_dy_f64", st);
  hipLaunchKernelGGL((k_dy_sum64<V>), dim3(blocks_for(rows * V::D_SH, 256)), dim3(256), 0, st, a.DY,
                     (const int*)nullptr, dy, rows, nsl);
  E3_HIP(hipGetLastError());
  return E3_OK;
}

template <class V>
e3_status run_fwd64(const e3_plan* p, const e3_graph* g, const double* x, const double* vec, const double* s,
                    double* m, hipStream_t st) {
  if (g->n_nodes == 0) return E3_OK;
  ConvArgs a = base_args(p, g);
  a.nslab = nslab64(p);
  const unsigned grid = (unsigned)(kXcd * a.chunk * V::NFG * a.nslab);
  TimedLaunch t_("conv_fwd_f64", st);
  hipLaunchKernelGGL((k_conv_fwd64<V>), dim3(grid), dim3(kWave), 0, st, a, x, vec, s, m);
  E3_HIP(hipGetLastError());
  return E3_OK;
}

template <class V>
e3_status run_bwd64(const e3_plan* p, const e3_graph* g, const double* x, const double* vec, const double* s,
                    const double* dm, double* dx, double* dvec, double* ds, void* ws, hipStream_t st) {
  if (g->n_nodes == 0) return E3_OK;
  const Ws w = bwd_ws64<V>(p, g);
  ConvArgs a = base_args(p, g);
  a.nslab = nslab64(p);
  Conv64Out o{x, vec, s, dm, ds, reinterpret_cast<double*>(ws),
              reinterpret_cast<double*>(reinterpret_cast<char*>(ws) + w.t_bytes)};
  if (g->n_live > 0) {
    const unsigned grid = (unsigned)(kXcd * a.chunk * V::NBG * a.nslab);
    TimedLaunch t_("conv_bwd_edges_f64", st);
    hipLaunchKernelGGL((k_conv_bwd64<V>), dim3(grid), dim3(kWave), 0, st, a, o);
    E3_HIP(hipGetLastError());
  }
  {
    TimedLaunch t_("conv_bwd_dx_f64", st);
    hipLaunchKernelGGL(k_conv_bwd_dx64, dim3((unsigned)(g->n_nodes * a.nslab)), dim3(kWave), 0, st, o.T, dx,
                       g->rowptr_s, a.n_nodes, V::D_IN, a.C, a.nslab);
    E3_HIP(hipGetLastError());
  }
  if (g->n_live > 0) {
    TimedLaunch t_("conv_bwd_dvec_f64", st);
    hipLaunchKernelGGL((k_conv_bwd_dvec64<V>), dim3(blocks_for(g->n_live, 256)), dim3(256), 0, st, vec, o.DY,
                       g->eid_r, dvec, g->n_live, a.nslab);
    E3_HIP(hipGetLastError());
  }
  if (g->n_pad > 0) {  // padding edges: zero ds and dvec rows (as pairs of 32-bit zeros)
    TimedLaunch t_("conv_bwd_pad", st);
    hipLaunchKernelGGL(k_zero_pad, dim3((unsigned)g->n_pad), dim3(256), 0, st, g->eid_r + g->n_live, g->n_pad,
                       reinterpret_cast<float*>(ds), (int64_t)2 * V::NP * a.C, reinterpret_cast<float*>(dvec),
                       (int64_t)6);
    E3_HIP(hipGetLastError());
  }
  return E3_OK;
}

// ---- launchers of a single-block kind (one channel per lane in the backward
// and tensor-product kernels; the accumulate flag is taken at run time)
template <class V>
e3_status kind_fwd(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* y,
                   const float* s, float* m, int accum, const KindCall& kc, hipStream_t st) {
  if (g->n_nodes == 0) return E3_OK;
  ConvArgs a = base_args(p, g);
  a.x = x, a.vec = vec, a.y = y, a.s = s, a.m = m, a.accum = accum;
  a.xr = kc.xr, a.pr = kc.pr, a.orr = kc.orr;
  a.nslab = p->nslab_f;
  const unsigned grid = (unsigned)(kXcd * a.chunk * V::NFG * a.nslab);
  {
    TimedLaunch t_("kind_fwd", st);
    if (p->cpl_f == 1)
      hipLaunchKernelGGL((k_conv_fwd<V, 1, false>), dim3(grid), dim3(kWave), 0, st, a);
    else
      hipLaunchKernelGGL((k_conv_fwd<V, E3_FWD_CPL, false>), dim3(grid), dim3(kWave), 0, st, a);
  }
  E3_HIP(hipGetLastError());
  return E3_OK;
}

template <class V>
e3_status kind_bwd(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* y,
                   const float* s, const float* dm, float* T, int64_t t_row, float* DY, float* ds, int64_t ds_row,
                   int accum_ds, const KindCall& kc, hipStream_t st) {
  if (g->n_live == 0) return E3_OK;
  ConvArgs a = base_args(p, g);
  a.x = x, a.vec = vec, a.y = y, a.s = s, a.dm = dm, a.accum = accum_ds;
  a.T = T, a.t_row = t_row, a.DY = DY, a.ds = ds, a.ds_row = ds_row;
  a.xr = kc.xr, a.pr = kc.pr, a.orr = kc.orr, a.ng = kc.ng, a.g0 = kc.g0;
  a.nslab = p->nslab_b;
  const unsigned grid = (unsigned)(kXcd * a.chunk * V::NBG * a.nslab);
  {
    TimedLaunch t_("kind_bwd", st);
    hipLaunchKernelGGL((k_conv_bwd_edges<V, 1, false>), dim3(grid), dim3(kWave), 0, st, a);
  }
  E3_HIP(hipGetLastError());
  return E3_OK;
}

template <class V>
e3_status kind_tp(const e3_plan* p, const float* x, const float* y, const float* w, float* z, int64_t rows,
                  const KindCall& kc, hipStream_t st) {
  if (rows == 0) return E3_OK;
  const int nslab = (p->lay.C + kWave - 1) / kWave;
  {
    TimedLaunch t_("kind_tp", st);
    const dim3 grid((unsigned)tile_grid(false, rows, kTpRows, nslab));
    hipLaunchKernelGGL((k_tp<V, 1>), grid, dim3(kWave), 0, st, x, y, w, z, rows, p->lay.C, nslab,
                       TpStr{kc.xr, kc.pr, kc.orr});
  }
  E3_HIP(hipGetLastError());
  return E3_OK;
}

template <class V>
e3_status kind_tpb(const e3_plan* p, const float* x, const float* y, const float* w, const float* dz, float* dx,
                   float* dw, float* DY, int64_t rows, const KindCall& kc, hipStream_t st) {
  if (rows == 0) return E3_OK;
  TpbArgs a{};
  a.x = x, a.y = y, a.w = w, a.dz = dz, a.dx = dx, a.dw = dw, a.DY = DY;
  a.rows = rows;
  a.C = p->lay.C;
  a.nslab = (a.C + kWave - 1) / kWave;
  a.xr = kc.xr, a.pr = kc.pr, a.orr = kc.orr, a.ng = kc.ng, a.g0 = kc.g0;
  {
    TimedLaunch t_("kind_tp_bwd", st);
    const dim3 grid((unsigned)tile_grid(E3_TP_XCD, rows, kTpRows, V::NBG * a.nslab));
    hipLaunchKernelGGL((k_tp_bwd<V, 1>), grid, dim3(kWave), 0, st, a);
  }
  E3_HIP(hipGetLastError());
  return E3_OK;
}

template <class V>
e3_status kind_fwd64(const e3_plan* p, const e3_graph* g, const double* x, const double* vec, const double* s,
                     double* m, const KindCall& kc, hipStream_t st) {
  if (g->n_nodes == 0) return E3_OK;
  ConvArgs a = base_args(p, g);
  a.nslab = nslab64(p);
  a.xr = kc.xr, a.pr = kc.pr, a.orr = kc.orr;
  const unsigned grid = (unsigned)(kXcd * a.chunk * V::NFG * a.nslab);
  TimedLaunch t_("kind_fwd_f64", st);
  hipLaunchKernelGGL((k_conv_fwd64<V>), dim3(grid), dim3(kWave), 0, st, a, x, vec, s, m);
  E3_HIP(hipGetLastError());
  return E3_OK;
}

template <class V>
e3_status kind_bwd64(const e3_plan* p, const e3_graph* g, const double* x, const double* vec, const double* s,
                     const double* dm, double* T, double* DY, double* ds, const KindCall& kc, hipStream_t st) {
  if (g->n_live == 0) return E3_OK;
  ConvArgs a = base_args(p, g);
  a.nslab = nslab64(p);
  a.xr = kc.xr, a.pr = kc.pr, a.orr = kc.orr, a.ng = kc.ng, a.g0 = kc.g0;
  Conv64Out o{x, vec, s, dm, ds, T, DY};
  const unsigned grid = (unsigned)(kXcd * a.chunk * V::NBG * a.nslab);
  TimedLaunch t_("kind_bwd_f64", st);
  hipLaunchKernelGGL((k_conv_bwd64<V>), dim3(grid), dim3(kWave), 0, st, a, o);
  E3_HIP(hipGetLastError());
  return E3_OK;
}

template <class V>
e3_status kind_tp64(const e3_plan* p, const double* x, const double* y, const double* w, double* z, int64_t rows,
                    const KindCall& kc, hipStream_t st) {
  if (rows == 0) return E3_OK;
  const int nsl = nslab64(p);
  const int64_t grid = tile_grid(false, rows, kBatch64, nsl);
  if (grid > 0x7fffffff) return E3_ERR_INVALID_ARG;
  TimedLaunch t_("kind_tp_f64", st);
  hipLaunchKernelGGL((k_tp64<V>), dim3((unsigned)grid), dim3(kWave), 0, st, x, y, w, z, rows, p->lay.C, nsl,
                     TpStr{kc.xr, kc.pr, kc.orr});
  E3_HIP(hipGetLastError());
  return E3_OK;
}

template <class V>
e3_status kind_tpb64(const e3_plan* p, const double* x, const double* y, const double* w, const double* dz,
                     double* dx, double* dw, double* DY, int64_t rows, const KindCall& kc, hipStream_t st) {
  if (rows == 0) return E3_OK;
  const int nsl = nslab64(p);
  Tpb64Args a{x, y, w, dz, dx, dw, DY, rows, p->lay.C, nsl, kc.xr, kc.pr, kc.orr, kc.ng, kc.g0};
  const int64_t grid = tile_grid(false, rows, kBatch64, V::NBG * nsl);
  if (grid > 0x7fffffff) return E3_ERR_INVALID_ARG;
  TimedLaunch t_("kind_tp_bwd_f64", st);
  hipLaunchKernelGGL((k_tp_bwd64<V>), dim3((unsigned)grid), dim3(kWave), 0, st, a);
  E3_HIP(hipGetLastError());
  return E3_OK;
}

template <class V>
e3_status kind_fwd_rad(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* h,
                       const float* W, int K, float* m, const KindCall& kc, hipStream_t st) {
  if (g->n_nodes == 0) return E3_OK;
  ConvArgs a = base_args(p, g);
  a.x = x, a.vec = vec, a.h = h, a.W = W, a.K = K, a.m = m;
  a.xr = kc.xr, a.pr = kc.pr, a.orr = kc.orr;
  a.nslab = p->nslab_b;
  const unsigned grid = (unsigned)(kXcd * a.chunk * V::NFG * a.nslab);
  {
    TimedLaunch t_("kind_fwd_rad", st);
    if (K <= 8 && E3_RAD_WREG)
      hipLaunchKernelGGL((k_conv_fwd_rad<V, 8>), dim3(grid), dim3(kWave), 0, st, a);
    else
      hipLaunchKernelGGL((k_conv_fwd_rad<V, 0>), dim3(grid), dim3(kWave), 0, st, a);
  }
  E3_HIP(hipGetLastError());
  return E3_OK;
}

template <class V>
e3_status kind_bwd_rad(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* h,
                       const float* W, int K, const float* dm, float* T, float* DY, float* DS, const KindCall& kc,
                       hipStream_t st) {
  if (g->n_live == 0) return E3_OK;
  ConvArgs a = base_args(p, g);
  a.x = x, a.vec = vec, a.h = h, a.W = W, a.K = K, a.dm = dm, a.T = T, a.DY = DY, a.ds = DS;
  a.xr = kc.xr, a.pr = kc.pr, a.orr = kc.orr, a.ng = kc.ng, a.g0 = kc.g0;
  a.nslab = p->nslab_b;
  const unsigned grid = (unsigned)(kXcd * a.chunk * V::NBG * a.nslab);
  TimedLaunch t_("kind_bwd_rad", st);
  hipLaunchKernelGGL((k_conv_bwd_rad<V>), dim3(grid), dim3(kWave), 0, st, a);
  E3_HIP(hipGetLastError());
  return E3_OK;
}

template <class V>
e3_status kind_fwd3(const e3_plan* p, const e3_graph* g, const float* x, const float* x2, const float* y,
                    const float* y2, const float* s, const float* s2, float* m, const KindCall& kc, hipStream_t st) {
  if (g->n_nodes == 0) return E3_OK;
  ConvArgs a = base_args(p, g);
  a.x = x, a.x2 = x2, a.y = y, a.y2 = y2, a.s = s, a.s2 = s2, a.m = m;
  a.xr = kc.xr, a.pr = kc.pr, a.orr = kc.orr;
  fwd3_slabs(a);
  const unsigned grid = (unsigned)(kXcd * a.chunk * V::NFG * a.nslab);
  TimedLaunch t_("kind_fwd3", st);
  hipLaunchKernelGGL((k_conv_fwd3<V>), dim3(grid), dim3(a.sw * kWave), fwd3_lds_bytes<V>(a), st, a);
  E3_HIP(hipGetLastError());
  return E3_OK;
}

template <class V>
e3_status kind_bwd3(const e3_plan* p, const e3_graph* g, const float* x, const float* x2, const float* y,
                    const float* y2, const float* s, const float* s2, const float* dm, float* T, float* DY,
                    float* gs, const KindCall& kc, hipStream_t st) {
  if (g->n_live == 0) return E3_OK;
  ConvArgs a = base_args(p, g);
  a.x = x, a.x2 = x2, a.y = y, a.y2 = y2, a.s = s, a.s2 = s2, a.dm = dm, a.ds = gs, a.T = T, a.DY = DY;
  a.xr = kc.xr, a.pr = kc.pr, a.orr = kc.orr, a.ng = kc.ng, a.g0 = kc.g0;
  a.nslab = p->nslab_b;
  const unsigned grid = (unsigned)(kXcd * a.chunk * V::NBG * a.nslab);
  TimedLaunch t_("kind_bwd3", st);
  hipLaunchKernelGGL((k_conv_bwd3<V>), dim3(grid), dim3(kWave), 0, st, a);
  E3_HIP(hipGetLastError());
  return E3_OK;
}

}  // namespace

// One kind's entry in the composed path's table (constant-initialised).
#define E3_KIND_OPS(V)                                                                                  \
  KindOps{e3gen::V::SIG, e3gen::V::D_IN, e3gen::V::D_SH, e3gen::V::D_OUT, e3gen::V::NP, e3gen::V::LSH, \
          e3gen::V::NBG, &kind_fwd<e3gen::V>, &kind_bwd<e3gen::V>, &kind_tp<e3gen::V>,                 \
          &kind_tpb<e3gen::V>, &kind_fwd64<e3gen::V>, &kind_bwd64<e3gen::V>, &kind_tp64<e3gen::V>,     \
          &kind_tpb64<e3gen::V>, &kind_fwd_rad<e3gen::V>, &kind_bwd_rad<e3gen::V>, &kind_fwd3<e3gen::V>,  \
          &kind_bwd3<e3gen::V>}

// One variant's entry in the core unit's table (constant-initialised).
#define E3_VARIANT_OPS(V)                                                                                    \
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
             &run_bwd3<e3gen::V>,                                                                        \
             &run_tp64<e3gen::V>,                                                                        \
             &run_tp_bwd64<e3gen::V>,                                                                    \
             &tp_ws64<e3gen::V>,                                                                         \
             &run_fwd64<e3gen::V>,                                                                       \
             &run_bwd64<e3gen::V>,                                                                       \
             &bwd_ws64<e3gen::V>}
