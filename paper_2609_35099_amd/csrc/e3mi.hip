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

#include "e3mi_impl.h"

// ------------------------------------------------------------ shared state
thread_local std::string g_last_error;
Timing g_timing;

// The compiled variants, each defined in its own unit (generated list).
#include "generated/variant_table.inc"

namespace {
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
                             int* __restrict__ bad) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= n_edges) return;
  const int32_t s = snd[e], r = rcv[e];
  const bool out_of_range = s < 0 || s >= n_nodes || r < 0 || r >= n_nodes;
  if (out_of_range) *bad = 1;  // every writer stores the same value
  // an out-of-range index becomes the padding key (the build fails anyway),
  // so that the sort's digits stay below 2^bits
  const bool is_pad = out_of_range || (pad >= 0 && (s == pad || r == pad));
  key_r[e] = is_pad ? (uint32_t)n_nodes : (uint32_t)r;
  key_s[e] = is_pad ? (uint32_t)n_nodes : (uint32_t)s;
}

// Stable LSD radix sort of (key, edge id) pairs, 8 bits of the key per pass.
// A tile is kSortRounds rounds of one 256-thread block over consecutive
// elements.  Per pass: k_sort_hist counts each tile's digits, k_sort_scan turns
// each digit's tile counts into exclusive offsets and a digit total, and
// k_sort_scatter places every element at
//   (elements of smaller digits) + offset[digit][tile]
//   + (same-digit elements of earlier rounds of its tile)
//   + (same-digit elements of earlier waves of its round)
//   + (same-digit elements of lower lanes of its wave),
// so equal digits keep their input order and every pass is stable.  Integer
// counts only: the result does not depend on scheduling.
constexpr int kSortBlock = 256, kSortRounds = 16, kSortTile = kSortBlock * kSortRounds;
constexpr int kSortWaves = kSortBlock / kWave;
static_assert(kSortBlock == 256, "one thread per digit");

__global__ __launch_bounds__(kSortBlock) void k_sort_hist(const uint32_t* __restrict__ keys, int64_t n, int shift,
                                                          int64_t n_tiles, int32_t* __restrict__ count) {
  __shared__ int hist[256];
  const int tid = threadIdx.x;
  hist[tid] = 0;
  __syncthreads();
  const int64_t t = blockIdx.x;
  for (int j = 0; j < kSortRounds; ++j) {
    const int64_t i = t * kSortTile + (int64_t)j * kSortBlock + tid;
    if (i < n) atomicAdd(&hist[(keys[i] >> shift) & 255u], 1);
  }
  __syncthreads();
  count[(int64_t)tid * n_tiles + t] = hist[tid];
}

// Inclusive scan of v over the block (Hillis-Steele in LDS); total = the sum
// over the block.  Ends with a barrier after the last reads of buf.
__device__ __forceinline__ int32_t block_incl_scan(int32_t v, int32_t (&buf)[2][kSortBlock], int tid,
                                                   int32_t& total) {
  buf[0][tid] = v;
  __syncthreads();
  int cur = 0;
  for (int d = 1; d < kSortBlock; d <<= 1) {
    const int32_t u = buf[cur][tid] + (tid >= d ? buf[cur][tid - d] : 0);
    buf[cur ^ 1][tid] = u;
    cur ^= 1;
    __syncthreads();
  }
  const int32_t incl = buf[cur][tid];
  total = buf[cur][kSortBlock - 1];
  __syncthreads();
  return incl;
}

// Per digit (one block each): exclusive scan of its tiles' counts in place
// (row d of count) and the digit's total.
__global__ __launch_bounds__(kSortBlock) void k_sort_scan(int32_t* __restrict__ count, int64_t n_tiles,
                                                          int32_t* __restrict__ total) {
  __shared__ int32_t buf[2][kSortBlock];
  const int tid = threadIdx.x;
  int32_t* row = count + (int64_t)blockIdx.x * n_tiles;
  int32_t carry = 0;
  for (int64_t c0 = 0; c0 < n_tiles; c0 += kSortBlock) {
    const int64_t i = c0 + tid;
    const int32_t v = i < n_tiles ? row[i] : 0;
    int32_t chunk = 0;
    const int32_t incl = block_incl_scan(v, buf, tid, chunk);
    if (i < n_tiles) row[i] = carry + incl - v;
    carry += chunk;
  }
  if (tid == 0) total[blockIdx.x] = carry;
}

// ids_in == nullptr: the ids are the element indices.  Positions outside
// [0, n) cannot arise from consistent offsets; they are refused (bad = 1)
// rather than written.
__global__ __launch_bounds__(kSortBlock) void k_sort_scatter(const uint32_t* __restrict__ keys_in,
                                                             const int32_t* __restrict__ ids_in, int64_t n, int shift,
                                                             int64_t n_tiles, const int32_t* __restrict__ off,
                                                             const int32_t* __restrict__ total,
                                                             uint32_t* __restrict__ keys_out,
                                                             int32_t* __restrict__ ids_out, int* __restrict__ bad) {
  __shared__ int running[256];
  __shared__ int cnt[kSortWaves][256];
  __shared__ int32_t buf[2][kSortBlock];
  const int tid = threadIdx.x, lane = tid % kWave, w = tid / kWave;
  {
    // running starts at the digit's base: the elements of all smaller digits
    int32_t all = 0;
    const int32_t v = total[tid];
    running[tid] = block_incl_scan(v, buf, tid, all) - v;
  }
#pragma unroll
  for (int k = 0; k < kSortWaves; ++k) cnt[k][tid] = 0;
  __syncthreads();
  const int64_t t = blockIdx.x;
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (kWave - lane));
  for (int j = 0; j < kSortRounds; ++j) {
    const int64_t i = t * kSortTile + (int64_t)j * kSortBlock + tid;
    const bool valid = i < n;
    const uint32_t key = valid ? keys_in[i] : 0u;
    const int32_t id = valid ? (ids_in ? ids_in[i] : (int32_t)i) : 0;
    const int d = (int)((key >> shift) & 255u);
    // lanes of this wave holding the same digit
    uint64_t same = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const uint64_t set = __ballot(valid && ((d >> bit) & 1));
      same &= ((d >> bit) & 1) ? set : ~set;
    }
    const int rank = __popcll(same & below);
    if (valid && (same & below) == 0) cnt[w][d] = __popcll(same);  // the digit's lowest lane
    __syncthreads();
    if (valid) {
      int prefix = 0;
      for (int k = 0; k < w; ++k) prefix += cnt[k][d];
      const int64_t pos = (int64_t)off[(int64_t)d * n_tiles + t] + running[d] + prefix + rank;
      if (pos >= 0 && pos < n) {
        keys_out[pos] = key;
        ids_out[pos] = id;
      } else {
        *bad = 1;
      }
    }
    __syncthreads();
    int add = 0;
#pragma unroll
    for (int k = 0; k < kSortWaves; ++k) add += cnt[k][tid], cnt[k][tid] = 0;
    running[tid] += add;
    __syncthreads();
  }
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

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int cpl_index(int cpl) { return cpl == 1 ? 0 : 1; }
int cpl_of(const e3_plan* p) { return p->cpl_f; }

// A compiled variant (every entry point).
e3_status check_plan(const e3_plan* p) {
  if (!p) return E3_ERR_INVALID_ARG;
  if (p->variant < 0) {
    g_last_error = p->rec ? "this entry point needs a compiled kernel variant for the layout"
                          : p->no_rec_reason;
    return E3_ERR_UNSUPPORTED;
  }
  return E3_OK;
}

// A compiled variant, or the record path with its tables on the current
// device (the convolution and tensor-product forward and backward).
e3_status check_any(const e3_plan* p) {
  if (!p) return E3_ERR_INVALID_ARG;
  return p->variant >= 0 ? E3_OK : rec_check(p);
}

// A compiled variant or the composed path (the float64 builds and the fused
// radial weights, which the record path does not have).
e3_status check_composable(const e3_plan* p) {
  if (!p) return E3_ERR_INVALID_ARG;
  if (p->variant >= 0 || p->composed) return E3_OK;
  g_last_error = p->rec ? "this entry point needs a compiled variant or the composed path" : p->no_rec_reason;
  return E3_ERR_UNSUPPORTED;
}

Ws conv_ws(const e3_plan* p, const e3_graph* g) {
  return p->variant >= 0 ? (*kVariants[p->variant]()).ws(p, g) : rec_ws(p, g);
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
  if (lmax_sh < 0 || lmax_sh > 3 || lmax_out < 0 || lmax_out > 16 ||
      (flags & ~(E3_PARITY_NATURAL | E3_PLAN_RECORDS | E3_PLAN_COMPOSED)) ||
      ((flags & E3_PLAN_RECORDS) && (flags & E3_PLAN_COMPOSED)))
    return E3_ERR_INVALID_ARG;
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
  if (!e3b::make_layout(irreps_x, lmax_sh, lmax_out, (flags & E3_PARITY_NATURAL) != 0, p->lay, err)) {
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
  if (C >= 4 && C % 4 == 0 && C <= kMaxChannels && !(flags & (E3_PLAN_RECORDS | E3_PLAN_COMPOSED))) {
    for (int i = 0; i < kNumVariants; ++i)
      if (sig == kVariants[i]()->sig && p->lay.d_sh == kVariants[i]()->d_sh) p->variant = i;
  }
  if (p->variant >= 0) {
    p->cpl_f = C <= kWave ? 1 : E3_FWD_CPL;
    p->nslab_f = (C + kWave * p->cpl_f - 1) / (kWave * p->cpl_f);
    p->cpl_b = C <= kWave ? 1 : E3_BWD_CPL;
    p->nslab_b = (C + kWave * p->cpl_b - 1) / (kWave * p->cpl_b);
  } else if ((flags & E3_PLAN_RECORDS) || comp_create(p) != E3_OK) {
    // still a valid plan (its tables can be queried) when neither path takes
    // it: its compute calls report why
    if (flags & E3_PLAN_COMPOSED)
      p->no_rec_reason = "the composed path takes x blocks and outputs of degree <= 3 and C a multiple of 4 "
                         "up to " + std::to_string(kMaxChannels);
    else if (rec_create(p) != E3_OK)
      p->no_rec_reason = g_last_error;
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
  info->supported = p->variant >= 0 ? 1 : p->composed ? 3 : (rec_ready(p) ? 2 : 0);
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

namespace {
// Stable sort of keys[0, n) < 2^nbits with their element indices as ids:
// ceil(nbits / 8) passes ping-ponging between (tk, ti) and the outputs, so that
// the last lands in (keys_out, ids_out).  count holds 256 * (tiles + 1) ints
// (the tile counts, then the digit totals).
hipError_t sort_pairs(const uint32_t* keys, int64_t n, int nbits, uint32_t* keys_out, int32_t* ids_out,
                      uint32_t* tk, int32_t* ti, int32_t* count, int* bad, hipStream_t st) {
  const int64_t tiles = (n + kSortTile - 1) / kSortTile;
  const int passes = (nbits + 7) / 8;
  const uint32_t* kin = keys;
  const int32_t* iin = nullptr;
  for (int p = 0; p < passes; ++p) {
    const bool to_out = ((passes - 1 - p) % 2) == 0;
    uint32_t* kout = to_out ? keys_out : tk;
    int32_t* iout = to_out ? ids_out : ti;
    hipLaunchKernelGGL(k_sort_hist, dim3((unsigned)tiles), dim3(kSortBlock), 0, st, kin, n, 8 * p, tiles, count);
    hipLaunchKernelGGL(k_sort_scan, dim3(256), dim3(kSortBlock), 0, st, count, tiles, count + 256 * tiles);
    hipLaunchKernelGGL(k_sort_scatter, dim3((unsigned)tiles), dim3(kSortBlock), 0, st, kin, iin, n, 8 * p, tiles,
                       count, count + 256 * tiles, kout, iout, bad);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    kin = kout, iin = iout;
  }
  return hipSuccess;
}
}  // namespace

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
  uint32_t *key_r = nullptr, *key_s = nullptr, *key_sorted = nullptr, *tk = nullptr;
  int32_t *ti = nullptr, *count = nullptr;
  int* flag = nullptr;
  auto cleanup = [&]() {
    (void)hipFree(key_r), (void)hipFree(key_s), (void)hipFree(key_sorted), (void)hipFree(tk), (void)hipFree(ti),
        (void)hipFree(count), (void)hipFree(flag);
  };
  const int64_t tiles = (E + kSortTile - 1) / kSortTile;
  if (!alloc((void**)&key_r, E * 4) || !alloc((void**)&key_s, E * 4) || !alloc((void**)&key_sorted, E * 4) ||
      !alloc((void**)&tk, E * 4) || !alloc((void**)&ti, E * 4) || !alloc((void**)&count, 256 * (tiles + 1) * 4) ||
      !alloc((void**)&flag, 2 * sizeof(int))) {
    cleanup();
    return fail(E3_ERR_ALLOC);
  }
  // keys are receivers (senders) in [0, N), padding edges N
  int end_bit = 1;
  while (end_bit < 32 && ((int64_t)1 << end_bit) <= N) ++end_bit;
  hipError_t herr = hipSuccess;
  herr = hipMemsetAsync(flag, 0, 2 * sizeof(int), st);
  if (herr == hipSuccess && E > 0) {
    hipLaunchKernelGGL(k_graph_keys, dim3(blocks_for(E, 256)), dim3(256), 0, st, sender, receiver, E, (int32_t)N,
                       pad_node, key_r, key_s, flag);
    herr = hipGetLastError();
    if (herr == hipSuccess)
      herr = sort_pairs(key_r, E, end_bit, key_sorted, g->eid_r, tk, ti, count, flag + 1, st);
    if (herr == hipSuccess) {
      hipLaunchKernelGGL(k_graph_rowptr, dim3(blocks_for(N + 1, 256)), dim3(256), 0, st, key_sorted, E, (int32_t)N,
                         g->rowptr_r);
      herr = hipGetLastError();
    }
    if (herr == hipSuccess)
      herr = sort_pairs(key_s, E, end_bit, key_sorted, g->eid_s, tk, ti, count, flag + 1, st);
    if (herr == hipSuccess) {
      hipLaunchKernelGGL(k_graph_rowptr, dim3(blocks_for(N + 1, 256)), dim3(256), 0, st, key_sorted, E, (int32_t)N,
                         g->rowptr_s);
      herr = hipGetLastError();
    }
  } else if (herr == hipSuccess) {
    herr = hipMemsetAsync(g->rowptr_r, 0, (N + 1) * 4, st);
    if (herr == hipSuccess) herr = hipMemsetAsync(g->rowptr_s, 0, (N + 1) * 4, st);
  }
  int host[3] = {0, 0, 0};
  if (herr == hipSuccess) herr = hipMemcpyAsync(&host[0], flag, 2 * sizeof(int), hipMemcpyDeviceToHost, st);
  if (herr == hipSuccess) herr = hipMemcpyAsync(&host[2], g->rowptr_r + N, sizeof(int), hipMemcpyDeviceToHost, st);
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
  if (host[1]) {
    g_last_error = "e3_graph_create: inconsistent sort offsets";
    cleanup();
    return fail(E3_ERR_HIP);
  }
  g->n_live = host[2];
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
  e3_status s = check_any(p);
  if (s != E3_OK) return s;
  if (rows < 0) return E3_ERR_INVALID_ARG;
  if (rows > 0 && (!x || !y || !w || !z || !aligned16(x) || !aligned16(w) || !aligned16(z))) return E3_ERR_INVALID_ARG;
  if (rows == 0) return E3_OK;
  if (p->variant < 0) return rec_fwd(p, nullptr, rows, x, nullptr, y, w, z, 0, reinterpret_cast<hipStream_t>(stream));
  const VariantOps& v = (*kVariants[p->variant]());
  return v.tp[cpl_index(cpl_of(p))](p, x, y, w, z, rows, reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_tp_workspace_size(const e3_plan* p, int64_t rows, size_t* bwd_bytes) {
  e3_status s = check_any(p);
  if (s != E3_OK) return s;
  if (rows < 0 || !bwd_bytes) return E3_ERR_INVALID_ARG;
  *bwd_bytes = p->variant >= 0 ? (*kVariants[p->variant]()).tpws(p, rows) : rec_tp_ws(p, rows);
  return E3_OK;
}

e3_status e3_tp_bwd(const e3_plan* p, const float* x, const float* y, const float* w, const float* dz, float* dx,
                    float* dy, float* dw, void* ws, size_t ws_bytes, int64_t rows, e3_stream stream) {
  e3_status s = check_any(p);
  if (s != E3_OK) return s;
  if (rows < 0) return E3_ERR_INVALID_ARG;
  if (rows == 0) return E3_OK;
  if (!x || !y || !w || !dz || !dx || !dy || !dw || !ws || !aligned16(x) || !aligned16(w) || !aligned16(dz) ||
      !aligned16(dx) || !aligned16(dw) || !aligned16(ws))
    return E3_ERR_INVALID_ARG;
  if (p->variant < 0) {
    if (ws_bytes < rec_tp_ws(p, rows)) return E3_ERR_WORKSPACE_TOO_SMALL;
    return rec_bwd(p, nullptr, rows, x, nullptr, y, w, dz, dx, nullptr, dy, dw, 0, ws,
                   reinterpret_cast<hipStream_t>(stream));
  }
  const VariantOps& v = (*kVariants[p->variant]());
  if (ws_bytes < v.tpws(p, rows)) return E3_ERR_WORKSPACE_TOO_SMALL;
  return v.tpb(p, x, y, w, dz, dx, dy, dw, ws, rows, reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_conv_workspace_size(const e3_plan* p, const e3_graph* g, size_t* fwd_bytes, size_t* bwd_bytes) {
  e3_status s = check_any(p);
  if (s != E3_OK) return s;
  if (!g) return E3_ERR_INVALID_ARG;
  Ws w = conv_ws(p, g);
  if (fwd_bytes) *fwd_bytes = 0;
  if (bwd_bytes) *bwd_bytes = w.t_bytes + w.dy_bytes;
  return E3_OK;
}

e3_status e3_conv_fwd(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* s,
                      float* m, void* ws, size_t ws_bytes, e3_stream stream) {
  (void)ws, (void)ws_bytes;
  e3_status st = check_any(p);
  if (st != E3_OK) return st;
  if (!g) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!m || !aligned16(m) || !x || !aligned16(x))) return E3_ERR_INVALID_ARG;
  if (g->n_live > 0 && (!vec || !s || !aligned16(s))) return E3_ERR_INVALID_ARG;
  if (p->variant < 0) return rec_fwd(p, g, 0, x, vec, nullptr, s, m, 0, reinterpret_cast<hipStream_t>(stream));
  const VariantOps& v = (*kVariants[p->variant]());
  return v.fwd[cpl_index(cpl_of(p))](p, g, x, vec, nullptr, s, m, 0, reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_conv_bwd(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* s,
                      const float* dm, float* dx, float* dvec, float* ds, void* ws, size_t ws_bytes,
                      e3_stream stream) {
  e3_status st = check_any(p);
  if (st != E3_OK) return st;
  if (!g) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!x || !dm || !dx || !aligned16(x) || !aligned16(dm) || !aligned16(dx)))
    return E3_ERR_INVALID_ARG;
  if (g->n_edges > 0 && (!vec || !s || !ds || !dvec || !aligned16(s) || !aligned16(ds))) return E3_ERR_INVALID_ARG;
  Ws w = conv_ws(p, g);
  if (w.t_bytes + w.dy_bytes > 0 && (!ws || !aligned16(ws))) return E3_ERR_INVALID_ARG;
  if (ws_bytes < w.t_bytes + w.dy_bytes) return E3_ERR_WORKSPACE_TOO_SMALL;
  if (p->variant < 0)
    return rec_bwd(p, g, 0, x, vec, nullptr, s, dm, dx, dvec, nullptr, ds, 0, ws,
                   reinterpret_cast<hipStream_t>(stream));
  const VariantOps& v = (*kVariants[p->variant]());
  return v.bwd[cpl_index(cpl_of(p))](p, g, x, vec, nullptr, s, dm, dx, dvec, nullptr, ds, 0, ws,
                                     reinterpret_cast<hipStream_t>(stream));
}

// ---- float64 builds
e3_status e3_tp_fwd_f64(const e3_plan* p, const double* x, const double* y, const double* w, double* z,
                        int64_t rows, e3_stream stream) {
  e3_status s = check_composable(p);
  if (s != E3_OK) return s;
  if (rows < 0) return E3_ERR_INVALID_ARG;
  if (rows == 0) return E3_OK;
  if (!x || !y || !w || !z || !aligned16(x) || !aligned16(w) || !aligned16(z)) return E3_ERR_INVALID_ARG;
  if (p->variant < 0) return comp_tp64(p, x, y, w, z, rows, reinterpret_cast<hipStream_t>(stream));
  return (*kVariants[p->variant]()).tp64(p, x, y, w, z, rows, reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_tp_workspace_size_f64(const e3_plan* p, int64_t rows, size_t* bwd_bytes) {
  e3_status s = check_composable(p);
  if (s != E3_OK) return s;
  if (rows < 0 || !bwd_bytes) return E3_ERR_INVALID_ARG;
  *bwd_bytes = p->variant >= 0 ? (*kVariants[p->variant]()).tpws64(p, rows) : comp_tp_ws64(p, rows);
  return E3_OK;
}

e3_status e3_tp_bwd_f64(const e3_plan* p, const double* x, const double* y, const double* w, const double* dz,
                        double* dx, double* dy, double* dw, void* ws, size_t ws_bytes, int64_t rows,
                        e3_stream stream) {
  e3_status s = check_composable(p);
  if (s != E3_OK) return s;
  if (rows < 0) return E3_ERR_INVALID_ARG;
  if (rows == 0) return E3_OK;
  if (!x || !y || !w || !dz || !dx || !dy || !dw || !ws || !aligned16(x) || !aligned16(w) || !aligned16(dz) ||
      !aligned16(dx) || !aligned16(dw) || !aligned16(ws))
    return E3_ERR_INVALID_ARG;
  if (p->variant < 0) {
    if (ws_bytes < comp_tp_ws64(p, rows)) return E3_ERR_WORKSPACE_TOO_SMALL;
    return comp_tpb64(p, x, y, w, dz, dx, dy, dw, ws, rows, reinterpret_cast<hipStream_t>(stream));
  }
  const VariantOps& v = (*kVariants[p->variant]());
  if (ws_bytes < v.tpws64(p, rows)) return E3_ERR_WORKSPACE_TOO_SMALL;
  return v.tpb64(p, x, y, w, dz, dx, dy, dw, ws, rows, reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_conv_workspace_size_f64(const e3_plan* p, const e3_graph* g, size_t* bwd_bytes) {
  e3_status s = check_composable(p);
  if (s != E3_OK) return s;
  if (!g || !bwd_bytes) return E3_ERR_INVALID_ARG;
  const Ws w = p->variant >= 0 ? (*kVariants[p->variant]()).ws64(p, g) : comp_ws64(p, g);
  *bwd_bytes = w.t_bytes + w.dy_bytes;
  return E3_OK;
}

e3_status e3_conv_fwd_f64(const e3_plan* p, const e3_graph* g, const double* x, const double* vec, const double* s,
                          double* m, e3_stream stream) {
  e3_status st = check_composable(p);
  if (st != E3_OK) return st;
  if (!g) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!x || !m || !aligned16(x) || !aligned16(m))) return E3_ERR_INVALID_ARG;
  if (g->n_edges > 0 && (!vec || !s || !aligned16(s))) return E3_ERR_INVALID_ARG;
  if (p->variant < 0) return comp_fwd64(p, g, x, vec, s, m, reinterpret_cast<hipStream_t>(stream));
  return (*kVariants[p->variant]()).fwd64(p, g, x, vec, s, m, reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_conv_bwd_f64(const e3_plan* p, const e3_graph* g, const double* x, const double* vec, const double* s,
                          const double* dm, double* dx, double* dvec, double* ds, void* ws, size_t ws_bytes,
                          e3_stream stream) {
  e3_status st = check_composable(p);
  if (st != E3_OK) return st;
  if (!g) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!x || !dm || !dx || !aligned16(x) || !aligned16(dm) || !aligned16(dx)))
    return E3_ERR_INVALID_ARG;
  if (g->n_edges > 0 && (!vec || !s || !ds || !dvec || !aligned16(s) || !aligned16(ds))) return E3_ERR_INVALID_ARG;
  const Ws w = p->variant >= 0 ? (*kVariants[p->variant]()).ws64(p, g) : comp_ws64(p, g);
  if (w.t_bytes + w.dy_bytes > 0 && (!ws || !aligned16(ws))) return E3_ERR_INVALID_ARG;
  if (ws_bytes < w.t_bytes + w.dy_bytes) return E3_ERR_WORKSPACE_TOO_SMALL;
  if (p->variant < 0)
    return comp_bwd64(p, g, x, vec, s, dm, dx, dvec, ds, ws, reinterpret_cast<hipStream_t>(stream));
  return (*kVariants[p->variant]()).bwd64(p, g, x, vec, s, dm, dx, dvec, ds, ws,
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
  e3_status st = check_any(p);
  if (st != E3_OK) return st;
  if (!g) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!x || !dm || !dx || !aligned16(x) || !aligned16(dm) || !aligned16(dx)))
    return E3_ERR_INVALID_ARG;
  if (g->n_edges > 0 && (!vec || !s || !ds || !dvec || !aligned16(s) || !aligned16(ds))) return E3_ERR_INVALID_ARG;
  const Ws w = conv_ws(p, g);
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
  if (p->variant < 0)
    return rec_bwd(p, g, 0, x, vec, nullptr, s, dm, dx, dvec, nullptr, ds, 0, ptr,
                   reinterpret_cast<hipStream_t>(stream));
  const VariantOps& v = (*kVariants[p->variant]());
  return v.bwd[cpl_index(cpl_of(p))](p, g, x, vec, nullptr, s, dm, dx, dvec, nullptr, ds, 0, ptr,
                                     reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_conv_radial_workspace_size(const e3_plan* p, const e3_graph* g, int K, size_t* bwd_bytes) {
  e3_status st = check_composable(p);
  if (st != E3_OK) return st;
  if (!g || !bwd_bytes || K < 1 || K > kRadKMax) return E3_ERR_INVALID_ARG;
  *bwd_bytes = p->variant >= 0 ? (*kVariants[p->variant]()).rws(p, g, K).total() : comp_rad_ws(p, g, K).total();
  return E3_OK;
}

e3_status e3_conv_fwd_radial(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* h,
                             const float* W, int K, float* m, e3_stream stream) {
  e3_status st = check_composable(p);
  if (st != E3_OK) return st;
  if (!g || K < 1 || K > kRadKMax) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!m || !aligned16(m) || !x || !aligned16(x) || !W || !aligned16(W))) return E3_ERR_INVALID_ARG;
  if (g->n_live > 0 && (!vec || !h)) return E3_ERR_INVALID_ARG;
  if (p->variant < 0) return comp_fwd_rad(p, g, x, vec, h, W, K, m, reinterpret_cast<hipStream_t>(stream));
  return (*kVariants[p->variant]()).rfwd(p, g, x, vec, h, W, K, m, reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_conv_bwd_radial(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* h,
                             const float* W, int K, const float* dm, float* dx, float* dvec, float* dh, float* dW,
                             void* ws, size_t ws_bytes, e3_stream stream) {
  e3_status st = check_composable(p);
  if (st != E3_OK) return st;
  if (!g || K < 1 || K > kRadKMax || !W || !aligned16(W) || !dW) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!x || !dm || !dx || !aligned16(x) || !aligned16(dm) || !aligned16(dx)))
    return E3_ERR_INVALID_ARG;
  if (g->n_edges > 0 && (!vec || !h || !dh || !dvec)) return E3_ERR_INVALID_ARG;
  const RadWs w = p->variant >= 0 ? (*kVariants[p->variant]()).rws(p, g, K) : comp_rad_ws(p, g, K);
  if (w.total() > 0 && (!ws || !aligned16(ws))) return E3_ERR_INVALID_ARG;
  if (ws_bytes < w.total()) return E3_ERR_WORKSPACE_TOO_SMALL;
  if (p->variant < 0)
    return comp_bwd_rad(p, g, x, vec, h, W, K, dm, dx, dvec, dh, dW, ws, reinterpret_cast<hipStream_t>(stream));
  return (*kVariants[p->variant]()).rbwd(p, g, x, vec, h, W, K, dm, dx, dvec, dh, dW, ws,
                                         reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_conv_fwd_y(const e3_plan* p, const e3_graph* g, const float* x, const float* y, const float* s,
                        float* m, int accumulate, e3_stream stream) {
  e3_status st = check_any(p);
  if (st != E3_OK) return st;
  if (!g) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!m || !aligned16(m) || !x || !aligned16(x))) return E3_ERR_INVALID_ARG;
  if (g->n_live > 0 && (!y || !s || !aligned16(s))) return E3_ERR_INVALID_ARG;
  if (p->variant < 0)
    return rec_fwd(p, g, 0, x, nullptr, y, s, m, accumulate != 0, reinterpret_cast<hipStream_t>(stream));
  const VariantOps& v = (*kVariants[p->variant]());
  return v.fwd[cpl_index(cpl_of(p))](p, g, x, nullptr, y, s, m, accumulate != 0,
                                     reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_conv_bwd_y(const e3_plan* p, const e3_graph* g, const float* x, const float* y, const float* s,
                        const float* dm, float* dx, float* dy, float* ds, int accumulate, void* ws, size_t ws_bytes,
                        e3_stream stream) {
  e3_status st = check_any(p);
  if (st != E3_OK) return st;
  if (!g) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!x || !dm || !aligned16(x) || !aligned16(dm) || (dx && !aligned16(dx))))
    return E3_ERR_INVALID_ARG;
  if (g->n_edges > 0 && (!y || !s || !aligned16(s) || (ds && !aligned16(ds)))) return E3_ERR_INVALID_ARG;
  Ws w = conv_ws(p, g);
  if (w.t_bytes + w.dy_bytes > 0 && (!ws || !aligned16(ws))) return E3_ERR_INVALID_ARG;
  if (ws_bytes < w.t_bytes + w.dy_bytes) return E3_ERR_WORKSPACE_TOO_SMALL;
  if (p->variant < 0)
    return rec_bwd(p, g, 0, x, nullptr, y, s, dm, dx, nullptr, dy, ds, accumulate ? (kAccDx | kAccDy | kAccDs) : 0,
                   ws, reinterpret_cast<hipStream_t>(stream));
  const VariantOps& v = (*kVariants[p->variant]());
  return v.bwd[cpl_index(cpl_of(p))](p, g, x, nullptr, y, s, dm, dx, nullptr, dy, ds,
                                     accumulate ? (kAccDx | kAccDy | kAccDs) : 0, ws,
                                     reinterpret_cast<hipStream_t>(stream));
}

e3_status e3_conv_bwd2(const e3_plan* p, const e3_graph* g, const float* x, const float* y, const float* s,
                       const float* dm, const float* ddx, const float* ddy, const float* dds, float* gx, float* gy,
                       float* gs, float* gdm, void* ws, size_t ws_bytes, e3_stream stream) {
  e3_status st = check_any(p);
  if (st != E3_OK) return st;
  if (!g) return E3_ERR_INVALID_ARG;
  if (g->n_nodes > 0 && (!x || !dm || !ddx || !gx || !gdm || !aligned16(x) || !aligned16(dm) || !aligned16(ddx) ||
                         !aligned16(gx) || !aligned16(gdm)))
    return E3_ERR_INVALID_ARG;
  if (g->n_edges > 0 && (!y || !s || !ddy || !dds || !gy || !gs || !aligned16(s) || !aligned16(dds) ||
                         !aligned16(gs)))
    return E3_ERR_INVALID_ARG;
  Ws w = conv_ws(p, g);
  if (w.t_bytes + w.dy_bytes > 0 && (!ws || !aligned16(ws))) return E3_ERR_INVALID_ARG;
  if (ws_bytes < w.t_bytes + w.dy_bytes) return E3_ERR_WORKSPACE_TOO_SMALL;
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  if (p->composed) return comp_bwd2(p, g, x, y, s, dm, ddx, ddy, dds, gx, gy, gs, gdm, ws, hs);
  if (p->variant < 0) {  // the record path: three forward and three backward calls
    if ((st = rec_fwd(p, g, 0, ddx, nullptr, y, s, gdm, 0, hs)) != E3_OK) return st;
    if ((st = rec_fwd(p, g, 0, x, nullptr, ddy, s, gdm, 1, hs)) != E3_OK) return st;
    if ((st = rec_fwd(p, g, 0, x, nullptr, y, dds, gdm, 1, hs)) != E3_OK) return st;
    if ((st = rec_bwd(p, g, 0, ddx, nullptr, y, s, dm, nullptr, nullptr, gy, gs, 0, ws, hs)) != E3_OK) return st;
    if ((st = rec_bwd(p, g, 0, x, nullptr, ddy, s, dm, gx, nullptr, nullptr, gs, kAccDs, ws, hs)) != E3_OK)
      return st;
    return rec_bwd(p, g, 0, x, nullptr, y, dds, dm, gx, nullptr, gy, nullptr, kAccDx | kAccDy, ws, hs);
  }
  const VariantOps& v = (*kVariants[p->variant]());
  const int ci = cpl_index(cpl_of(p));
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
