// e3mi: the convolution and the weighted tensor product of layouts without a
// compiled variant (x blocks of degree <= 3, outputs to degree 3).  Two paths.
//
// The composed path (the default).  The build generates the kernels of every
// single x block kind -- degree, all or natural-parity paths, harmonics and
// output degrees -- with strides and offsets left to run time.  A layout runs
// block by block: each block's kernels read its x rows and path weights and
// write its output rows, its ds rows, its rows of the per-edge x-cotangent
// partials and its own harmonic partial groups; the sender-order segment sum
// and the fixed-order harmonic sum then finish the backward once.  Blocks
// without paths get zero cotangent rows.
//
// The record path (E3_PLAN_RECORDS): the same operations driven at run time
// by the plan's unfolded coupling records instead of code generated for the
// layout.  This is the paper's generic sparse kernel (App. E, "CUDA
// kernels": records (i0, i1, i2, value) over the whole unfolded axes, lanes
// on the trailing channels, one receiver's messages summed on chip over its
// receiver-CSR segment; App. E.2's trilinear form for the messages), run in
// this library's lane-per-channel layout.
//
// Work split.  The x blocks of the layout are cut into groups of consecutive
// whole blocks (at most 64 output rows, 16 x rows and 16 paths each); a wave
// takes one (receiver, group, 64-channel slab).  Whole blocks make the x
// cotangent rows of different groups disjoint, as in the compiled sweeps.
// Per batch of 8 edges the wave computes the harmonics and the group's
// pre-contraction A[pair] = sum_i2 C[i0, i1, i2] y[i2] over its (i0, i1)
// pairs into LDS; per edge it stages the sender's x rows and the edge's path
// weights in LDS and walks the pair lists.  Output rows are register
// accumulators (compile-time row slots, run-time row count); x rows, weights
// and pre-contraction entries are LDS reads at run-time addresses.
//
// The backward sweep follows eq. conv-bwd per edge: z = A x per output row
// gives ds[k] = sum over the rows of path k of z dm; w = s dm per row (kept in
// LDS); the x-cotangent partial t[i1] = sum_pairs A w (pairs by x row) goes
// to the same per-edge scratch as the compiled sweep, summed per sender by
// k_conv_bwd_dx; the harmonic cotangent dy[i2] = sum_records C x w (records
// by i2) is summed over the wave by the fixed tree and over groups and slabs
// in a fixed order, then mapped to dvec.  The tensor product is the same
// code on the identity graph (row r is edge r from node r to node r), with
// the x-cotangent partials stored straight into dx.
#include "e3mi_impl.h"
#include "generated/kind_table.inc"

namespace {

constexpr int kRecRows = 64, kRecX = 16, kRecPaths = 16, kRecBatch = 8;

// One group of whole x blocks; offsets into the int table.
struct RecGroup {
  int row0, nrows;    // output rows [row0, row0 + nrows)
  int pair0, npairs;  // its (i0, i1) pairs, a contiguous range in (i0, i1) order
  int x0, nx;         // x rows [x0, x0 + nx)
  int k0, npath;      // paths [k0, k0 + npath)
  int rowtab;         // nrows + 1 pair starts (relative to pair0), then per row: path-local index | last << 8
  int ttab;           // nx + 1 entry starts, then entries: pair-local | row-local << 16
  int dytab;          // D_sh + 1 entry starts (in entries), then entries: (x-local | row-local << 8, coefficient)
  int pad[5];
};
static_assert(sizeof(RecGroup) == 64, "group header");

struct RecArgs {
  const float* x;
  const float* vec;
  const float* y;
  const float* s;
  const float* dm;
  float* m;
  float* ds;
  float* T;
  float* DY;
  const int* rowptr;  // receiver CSR (null with ident)
  const int* eid;
  const int* src;
  const int* r2s;
  const RecGroup* grp;
  const int* tab;
  int o_pxl, o_prb, o_ri2, o_rc;  // table offsets: per pair x-local * 64, per pair record start, per record i2, value
  int n_nodes, chunk, C, nslab, ng, d_in, d_out, np, maxpairs, maxrows;
  int ident;  // the identity graph over n_nodes rows (the tensor product)
  int accum;  // forward: m += ; backward: ds +=
  int64_t ds_row, t_row;  // bytes of one ds / T block row set, 0: not stored
};

__device__ __forceinline__ bool rec_task(const RecArgs& a, int& b, int& g, int& sl) {
  const int bid = blockIdx.x;
  const int xcd = bid % kXcd, slot = bid / kXcd;
  const int per = a.ng * a.nslab;
  const int t = slot % per;
  g = t / a.nslab;
  sl = t % a.nslab;
  const int rl = slot / per;
  b = xcd * a.chunk + rl;
  return rl < a.chunk && b < a.n_nodes;
}

// Harmonics of the batch's edges (lane j < n: edge eb + j) into sY[j][16],
// then the group's pre-contraction of every edge of the batch into
// sA[j][maxpairs].  Lane j < n keeps its edge's id, sender and partial slot.
template <int LSH>
__device__ __forceinline__ void rec_batch(const RecArgs& a, ConstPtr<int> tab, int pair0, int npairs, int eb, int n,
                                          int& my_e, int& my_src, int& my_slot, float* sY, float* sA) {
  constexpr int DSH = (LSH + 1) * (LSH + 1);
  const int lane = threadIdx.x;
  if (lane < n) {
    const int pos = eb + lane;
    my_e = a.ident ? pos : a.eid[pos];
    my_src = a.ident ? pos : a.src[pos];
    my_slot = a.ident ? pos : (a.r2s ? a.r2s[pos] : 0);
    float Y[DSH];
    if (a.y) {
#pragma unroll
      for (int i = 0; i < DSH; ++i) Y[i] = a.y[(int64_t)my_e * DSH + i];
    } else {
      float ux, uy, uz, inv;
      unit_of(a.vec, my_e, ux, uy, uz, inv);
      sh_of<LSH>(ux, uy, uz, Y);
    }
#pragma unroll
    for (int i = 0; i < DSH; ++i) sY[lane * 16 + i] = Y[i];
  }
  __syncthreads();
  for (int idx = lane; idx < n * npairs; idx += kWave) {
    const int j = idx / npairs, pl = idx - j * npairs, p = pair0 + pl;
    const int r0 = tab[a.o_prb + p], r1 = tab[a.o_prb + p + 1];
    float v = 0.0f;
    for (int r = r0; r < r1; ++r) v = fmaf(__int_as_float(tab[a.o_rc + r]), sY[j * 16 + tab[a.o_ri2 + r]], v);
    sA[j * a.maxpairs + pl] = v;
  }
  __syncthreads();
}

// The sender's x rows and the edge's path weights of the group, one value per
// lane and row (rows past the group's counts and lanes past C hold zero).
struct RecStage {
  float xv[kRecX], sv[kRecPaths];
};

__device__ __forceinline__ void rec_load(const RecArgs& a, int64_t snd, int64_t e, int x0, int nx, int k0,
                                         int npath, int q, bool act, RecStage& st) {
  const int C = a.C;
#pragma unroll
  for (int i = 0; i < kRecX; ++i) st.xv[i] = 0.0f;
#pragma unroll
  for (int i = 0; i < kRecPaths; ++i) st.sv[i] = 0.0f;
  if (!act) return;
  // every access below is inside the group's rows of this node / edge
  const RowBuf xr = row_buf(a.x + (snd * a.d_in + x0) * C, (int64_t)nx * C * 4, q, C);
  const RowBuf sr = row_buf(a.s + (e * a.np + k0) * C, (int64_t)npath * C * 4, q, C);
#pragma unroll
  for (int i = 0; i < kRecX; ++i) {
    if (i < nx) {
      float v[1];
      bld<1>(xr, i, v);
      st.xv[i] = v[0];
    }
  }
#pragma unroll
  for (int i = 0; i < kRecPaths; ++i) {
    if (i < npath) {
      float v[1];
      bld<1, kNT>(sr, i, v);
      st.sv[i] = v[0];
    }
  }
}

__device__ __forceinline__ void rec_put(const RecStage& st, int nx, int npath, float* sX, float* sS) {
  const int lane = threadIdx.x;
#pragma unroll
  for (int i = 0; i < kRecX; ++i)
    if (i < nx) sX[i * kWave + lane] = st.xv[i];
#pragma unroll
  for (int i = 0; i < kRecPaths; ++i)
    if (i < npath) sS[i * kWave + lane] = st.sv[i];
}

// z of output row r of the group for the staged edge: sum over the row's
// pairs of A[pair] x[i1(pair)].
__device__ __forceinline__ float rec_row(const RecArgs& a, ConstPtr<int> tab, int pair0, int p0, int p1,
                                         const float* Aj, const float* sX) {
  const int lane = threadIdx.x;
  // two independent partial sums, added in a fixed order
  float z0 = 0.0f, z1 = 0.0f;
  int p = p0;
  for (; p + 2 <= p1; p += 2) {
    z0 = fmaf(Aj[p], sX[tab[a.o_pxl + pair0 + p] + lane], z0);
    z1 = fmaf(Aj[p + 1], sX[tab[a.o_pxl + pair0 + p + 1] + lane], z1);
  }
  if (p < p1) z0 = fmaf(Aj[p], sX[tab[a.o_pxl + pair0 + p] + lane], z0);
  return z0 + z1;
}

template <int LSH>
__global__ __launch_bounds__(kWave) void k_convr_fwd(RecArgs a) {
  extern __shared__ __align__(16) float lds[];
  int b, g, sl;
  if (!rec_task(a, b, g, sl)) return;
  const ConstPtr<int> tab = (ConstPtr<int>)a.tab;
  const ConstPtr<RecGroup> grp = (ConstPtr<RecGroup>)a.grp;
  const int row0 = grp[g].row0, nrows = grp[g].nrows, pair0 = grp[g].pair0, npairs = grp[g].npairs;
  const int x0 = grp[g].x0, nx = grp[g].nx, k0 = grp[g].k0, npath = grp[g].npath, rowtab = grp[g].rowtab;
  float* sY = lds;
  float* sA = sY + kRecBatch * 16;
  float* sX = sA + kRecBatch * a.maxpairs;
  float* sS = sX + kRecX * kWave;
  const int lane = threadIdx.x, C = a.C, q = sl * kWave + lane;
  const bool act = q < C;
  const int e0 = a.ident ? b : uniform(a.rowptr[b]), e1 = a.ident ? b + 1 : uniform(a.rowptr[b + 1]);
  float acc[kRecRows];
#pragma unroll
  for (int r = 0; r < kRecRows; ++r) acc[r] = 0.0f;
  for (int eb = e0; eb < e1; eb += kRecBatch) {
    const int n = imin(kRecBatch, e1 - eb);
    int my_e = 0, my_src = 0, my_slot = 0;
    rec_batch<LSH>(a, tab, pair0, npairs, eb, n, my_e, my_src, my_slot, sY, sA);
    RecStage st;
    rec_load(a, __builtin_amdgcn_readlane(my_src, 0), __builtin_amdgcn_readlane(my_e, 0), x0, nx, k0, npath, q,
             act, st);
    for (int j = 0; j < n; ++j) {
      rec_put(st, nx, npath, sX, sS);
      __syncthreads();
      if (j + 1 < n)  // the next edge's rows are in flight while this one computes
        rec_load(a, __builtin_amdgcn_readlane(my_src, j + 1), __builtin_amdgcn_readlane(my_e, j + 1), x0, nx, k0,
                 npath, q, act, st);
      const float* Aj = sA + j * a.maxpairs;
#pragma unroll
      for (int r = 0; r < kRecRows; ++r) {
        if (r < nrows) {
          const float z = rec_row(a, tab, pair0, tab[rowtab + r], tab[rowtab + r + 1], Aj, sX);
          const int kl = tab[rowtab + nrows + 1 + r] & 0xff;
          acc[r] = fmaf(sS[kl * kWave + lane], z, acc[r]);
        }
      }
      __syncthreads();
    }
  }
  if (act) {
    const RowBuf mb = row_buf(a.m + ((int64_t)b * a.d_out + row0) * C, (int64_t)nrows * C * 4, q, C);
#pragma unroll
    for (int r = 0; r < kRecRows; ++r) {
      if (r < nrows) {
        float v[1] = {acc[r]};
        if (a.accum) {
          float o[1];
          bld<1>(mb, r, o);
          v[0] += o[0];
        }
        bst<1, kST>(mb, r, v);
      }
    }
  }
}

template <int LSH>
__global__ __launch_bounds__(kWave) void k_convr_bwd(RecArgs a) {
  constexpr int DSH = (LSH + 1) * (LSH + 1);
  extern __shared__ __align__(16) float lds[];
  int b, g, sl;
  if (!rec_task(a, b, g, sl)) return;
  const int e0 = a.ident ? b : uniform(a.rowptr[b]), e1 = a.ident ? b + 1 : uniform(a.rowptr[b + 1]);
  if (e0 == e1) return;
  const ConstPtr<int> tab = (ConstPtr<int>)a.tab;
  const ConstPtr<RecGroup> grp = (ConstPtr<RecGroup>)a.grp;
  const int row0 = grp[g].row0, nrows = grp[g].nrows, pair0 = grp[g].pair0, npairs = grp[g].npairs;
  const int x0 = grp[g].x0, nx = grp[g].nx, k0 = grp[g].k0, npath = grp[g].npath, rowtab = grp[g].rowtab;
  const int ttab = grp[g].ttab, dytab = grp[g].dytab;
  float* sY = lds;
  float* sA = sY + kRecBatch * 16;
  float* sX = sA + kRecBatch * a.maxpairs;
  float* sS = sX + kRecX * kWave;
  float* sW = sS + kRecPaths * kWave;
  const int lane = threadIdx.x, C = a.C, q = sl * kWave + lane;
  const bool act = q < C;
  float dmv[kRecRows];
  {
    const RowBuf db = row_buf(a.dm + ((int64_t)b * a.d_out + row0) * C, (int64_t)nrows * C * 4, q, C);
#pragma unroll
    for (int r = 0; r < kRecRows; ++r) {
      float v[1] = {0.0f};
      if (act && r < nrows) bld<1>(db, r, v);
      dmv[r] = v[0];
    }
  }
  for (int eb = e0; eb < e1; eb += kRecBatch) {
    const int n = imin(kRecBatch, e1 - eb);
    int my_e = 0, my_src = 0, my_slot = 0;
    rec_batch<LSH>(a, tab, pair0, npairs, eb, n, my_e, my_src, my_slot, sY, sA);
    RecStage st;
    rec_load(a, __builtin_amdgcn_readlane(my_src, 0), __builtin_amdgcn_readlane(my_e, 0), x0, nx, k0, npath, q,
             act, st);
    for (int j = 0; j < n; ++j) {
      rec_put(st, nx, npath, sX, sS);
      __syncthreads();
      if (j + 1 < n)
        rec_load(a, __builtin_amdgcn_readlane(my_src, j + 1), __builtin_amdgcn_readlane(my_e, j + 1), x0, nx, k0,
                 npath, q, act, st);
      const int64_t e = __builtin_amdgcn_readlane(my_e, j);
      const int64_t slot = __builtin_amdgcn_readlane(my_slot, j);
      const float* Aj = sA + j * a.maxpairs;
      // z per row, ds per path (stored at the path's last row), w = s dm per row
      const RowBuf dsb = row_buf(a.ds + (e * a.np + k0) * C, a.ds_row ? (int64_t)npath * C * 4 : 0, q, C);
      float dsacc = 0.0f;
#pragma unroll
      for (int r = 0; r < kRecRows; ++r) {
        if (r < nrows) {
          const float z = rec_row(a, tab, pair0, tab[rowtab + r], tab[rowtab + r + 1], Aj, sX);
          const int info = tab[rowtab + nrows + 1 + r], kl = info & 0xff;
          dsacc = fmaf(z, dmv[r], dsacc);
          sW[r * kWave + lane] = sS[kl * kWave + lane] * dmv[r];
          if (info >> 8) {
            if (act) {
              float v[1] = {dsacc};
              if (a.accum) {
                float o[1];
                bld<1>(dsb, kl, o);
                v[0] += o[0];
              }
              bst<1, kST>(dsb, kl, v);
            }
            dsacc = 0.0f;
          }
        }
      }
      __syncthreads();
      // x-cotangent partials: t[i1] = sum over the pairs of x row i1 of A w
      {
        const RowBuf Tb = row_buf(a.T + (slot * a.d_in + x0) * C, a.t_row ? (int64_t)nx * C * 4 : 0, q, C);
#pragma unroll
        for (int xl = 0; xl < kRecX; ++xl) {
          if (xl < nx) {
            const int t0 = tab[ttab + xl], t1 = tab[ttab + xl + 1];
            // four independent partial sums, added in a fixed order
            float ta[4] = {0.0f, 0.0f, 0.0f, 0.0f};
            int u = t0;
            for (; u + 4 <= t1; u += 4) {
#pragma unroll
              for (int k = 0; k < 4; ++k) {
                const int ent = tab[ttab + nx + 1 + u + k];
                ta[k] = fmaf(Aj[ent & 0xffff], sW[(ent >> 16) * kWave + lane], ta[k]);
              }
            }
            for (; u < t1; ++u) {
              const int ent = tab[ttab + nx + 1 + u];
              ta[0] = fmaf(Aj[ent & 0xffff], sW[(ent >> 16) * kWave + lane], ta[0]);
            }
            float v[1] = {(ta[0] + ta[1]) + (ta[2] + ta[3])};
            if (act) bst<1, E3_T_STORE_AUX>(Tb, xl, v);
          }
        }
      }
      // harmonic cotangent of the lane's channel: dy[i2] = sum_records C x w
      float dyl[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) dyl[i] = 0.0f;
      const int dyent = dytab + DSH + 1;
#pragma unroll
      for (int i = 0; i < DSH; ++i) {
        const int u0 = tab[dytab + i], u1 = tab[dytab + i + 1];
        float va[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        int u = u0;
        for (; u + 4 <= u1; u += 4) {
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const int ent = tab[dyent + 2 * (u + k)];
            const float c = __int_as_float(tab[dyent + 2 * (u + k) + 1]);
            va[k] = fmaf(c, sX[(ent & 0xff) * kWave + lane] * sW[(ent >> 8) * kWave + lane], va[k]);
          }
        }
        for (; u < u1; ++u) {
          const int ent = tab[dyent + 2 * u];
          const float c = __int_as_float(tab[dyent + 2 * u + 1]);
          va[0] = fmaf(c, sX[(ent & 0xff) * kWave + lane] * sW[(ent >> 8) * kWave + lane], va[0]);
        }
        dyl[i] = (va[0] + va[1]) + (va[2] + va[3]);
      }
      const float tot = wave_reduce16(dyl, lane);
      if ((lane & 3) == 0) a.DY[(((int64_t)(eb + j) * a.ng + g) * a.nslab + sl) * 16 + (lane >> 2)] = tot;
      __syncthreads();
    }
  }
}

// dvec of each live edge from its harmonic cotangent, summed over the
// (group, slab) partials in order.
template <int LSH>
__global__ __launch_bounds__(256) void k_convr_dvec(const float* __restrict__ vec, const float* __restrict__ DY,
                                                    const int* __restrict__ eid, float* __restrict__ dvec,
                                                    int64_t n_live, int nparts) {
  constexpr int DSH = (LSH + 1) * (LSH + 1);
  const int64_t pos = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (pos >= n_live) return;
  const int64_t e = eid[pos];
  float dY[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) dY[i] = 0.0f;
  for (int g = 0; g < nparts; ++g)
#pragma unroll
    for (int i = 0; i < DSH; ++i) dY[i] += DY[(pos * nparts + g) * 16 + i];
  float ux, uy, uz, inv;
  unit_of(vec, e, ux, uy, uz, inv);
  float gx, gy, gz, ox, oy, oz;
  sh_grad_of<LSH>(ux, uy, uz, dY, gx, gy, gz);
  project(ux, uy, uz, inv, gx, gy, gz, ox, oy, oz);
  dvec[3 * e] = ox, dvec[3 * e + 1] = oy, dvec[3 * e + 2] = oz;
}

// dy of each live edge (eid null: position == row): the sum of its partials.
__global__ __launch_bounds__(256) void k_convr_dy(const float* __restrict__ DY, const int* __restrict__ eid,
                                                  float* __restrict__ dy, int64_t n_live, int dsh, int nparts,
                                                  int accum) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t r = i / dsh;
  const int c = (int)(i % dsh);
  if (r >= n_live) return;
  float v = 0.0f;
  for (int g = 0; g < nparts; ++g) v += DY[(r * nparts + g) * 16 + c];
  const int64_t o = (eid ? (int64_t)eid[r] : r) * dsh + c;
  dy[o] = accum ? dy[o] + v : v;
}

// Zero `len` floats at offset `off` of each of n rows of `stride` floats (the
// cotangent rows of x blocks without paths).
__global__ __launch_bounds__(256) void k_zero_rows(float* __restrict__ base, int64_t n, int64_t stride,
                                                   int64_t off, int64_t len) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n * len) return;
  base[(i / len) * stride + off + i % len] = 0.0f;
}

// float64: dvec of each live edge from its harmonic partials (summed in
// order), and dy (eid null: position == row).
template <int LSH>
__global__ __launch_bounds__(256) void k_convr_dvec64(const double* __restrict__ vec, const double* __restrict__ DY,
                                                      const int* __restrict__ eid, double* __restrict__ dvec,
                                                      int64_t n_live, int nparts) {
  constexpr int DSH = (LSH + 1) * (LSH + 1);
  const int64_t pos = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (pos >= n_live) return;
  const int64_t e = eid[pos];
  double dY[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) dY[i] = 0.0;
  for (int g = 0; g < nparts; ++g)
#pragma unroll
    for (int i = 0; i < DSH; ++i) dY[i] += DY[(pos * nparts + g) * 16 + i];
  double ux, uy, uz, inv, gx, gy, gz;
  unit_of64(vec, e, ux, uy, uz, inv);
  if constexpr (LSH == 0) e3gen::sh_grad_l0<double>(ux, uy, uz, dY, gx, gy, gz);
  else if constexpr (LSH == 1) e3gen::sh_grad_l1<double>(ux, uy, uz, dY, gx, gy, gz);
  else if constexpr (LSH == 2) e3gen::sh_grad_l2<double>(ux, uy, uz, dY, gx, gy, gz);
  else e3gen::sh_grad_l3<double>(ux, uy, uz, dY, gx, gy, gz);
  const double ug = ux * gx + uy * gy + uz * gz;
  dvec[3 * e] = (gx - ux * ug) * inv;
  dvec[3 * e + 1] = (gy - uy * ug) * inv;
  dvec[3 * e + 2] = (gz - uz * ug) * inv;
}

__global__ __launch_bounds__(256) void k_convr_dy64(const double* __restrict__ DY, const int* __restrict__ eid,
                                                    double* __restrict__ dy, int64_t n, int dsh, int nparts) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t r = i / dsh;
  const int c = (int)(i % dsh);
  if (r >= n) return;
  double v = 0.0;
  for (int g = 0; g < nparts; ++g) v += DY[(r * nparts + g) * 16 + c];
  dy[(eid ? (int64_t)eid[r] : r) * dsh + c] = v;
}

}  // namespace

// ============================================================ host
struct RecPlan {
  std::vector<RecGroup> groups;
  std::vector<int> tab;
  int o_pxl = 0, o_prb = 0, o_ri2 = 0, o_rc = 0;
  int maxpairs = 1, maxrows = 1, nslab = 1;
  int device = -1;
  char* dev = nullptr;  // groups, then the int table
};

e3_plan::~e3_plan() {
  if (rec) {
    if (rec->dev) (void)hipFree(rec->dev);
    delete rec;
  }
}

namespace {

// The record path's tables of a layout; false, with the reason in `why`, for
// a layout it does not take.
bool rec_tables(const e3_plan* p, RecPlan& R, std::string& why) {
  const auto& L = p->lay;
  if (L.C < 4 || L.C % 4 != 0 || L.C > kMaxChannels) {
    why = "channels must be a multiple of 4 up to " + std::to_string(kMaxChannels);
    return false;
  }
  if (L.lmax_out > 3) {
    why = "the record path takes output degrees up to 3";
    return false;
  }
  for (const auto& b : L.blocks)
    if (b.l > 3) {
      why = "the record path takes x blocks of degree up to 3";
      return false;
    }
  // pairs (i0, i1) in record order, the record range of each, and the first
  // pair of each output row
  std::vector<int> pi0, pi1, prb;
  for (size_t r = 0; r < p->recs.size(); ++r) {
    const auto& c = p->recs[r];
    if (pi0.empty() || pi0.back() != c.i0 || pi1.back() != c.i1) {
      pi0.push_back(c.i0), pi1.push_back(c.i1), prb.push_back((int)r);
    }
  }
  const int npair = (int)pi0.size(), nrec = (int)p->recs.size();
  prb.push_back(nrec);
  std::vector<int> row_pair(L.d_out + 1, npair);
  for (int pp = npair - 1; pp >= 0; --pp) row_pair[pi0[pp]] = pp;
  for (int i = L.d_out - 1; i >= 0; --i) row_pair[i] = std::min(row_pair[i], row_pair[i + 1]);
  // per x block: its x rows, paths and output rows
  const int nb = (int)L.blocks.size();
  std::vector<int> bx0(nb + 1, 0), bk0(nb + 1, 0), brow0(nb + 1, 0);
  for (int b = 0; b < nb; ++b) bx0[b + 1] = bx0[b] + 2 * L.blocks[b].l + 1;
  {
    int k = 0, row = 0;
    for (int b = 0; b < nb; ++b) {
      bk0[b] = k, brow0[b] = row;
      while (k < (int)L.paths.size() && L.paths[k].xb == b) row += 2 * L.paths[k].l3 + 1, ++k;
    }
    bk0[nb] = k, brow0[nb] = row;
    for (int kk = 0, rr = 0; kk < (int)L.paths.size(); rr += 2 * L.paths[kk].l3 + 1, ++kk)
      if (L.paths[kk].out_off != rr || L.paths[kk].x_off != bx0[L.paths[kk].xb]) k = -1;
    if (k != (int)L.paths.size() || row != L.d_out) {
      why = "paths are not ordered by x block with consecutive output rows";
      return false;
    }
  }
  // groups: consecutive whole blocks within the row, x-row and path limits
  std::vector<std::pair<int, int>> parts;
  for (int b = 0; b < nb;) {
    int e = b + 1;
    while (e < nb && brow0[e + 1] - brow0[b] <= kRecRows && bx0[e + 1] - bx0[b] <= kRecX &&
           bk0[e + 1] - bk0[b] <= kRecPaths)
      ++e;
    if (brow0[e] - brow0[b] > kRecRows || bx0[e] - bx0[b] > kRecX || bk0[e] - bk0[b] > kRecPaths) {
      why = "an x block exceeds the record path's per-wave limits";
      return false;
    }
    parts.push_back({b, e});
    b = e;
  }
  std::vector<int>& T = R.tab;
  R.o_pxl = (int)T.size();
  for (int pp = 0; pp < npair; ++pp) T.push_back(0);  // filled per group (x-local rows)
  R.o_prb = (int)T.size();
  for (int v : prb) T.push_back(v);
  R.o_ri2 = (int)T.size();
  for (const auto& c : p->recs) T.push_back(c.i2);
  R.o_rc = (int)T.size();
  for (const auto& c : p->recs) {
    const float f = (float)c.v;
    int bits;
    std::memcpy(&bits, &f, 4);
    T.push_back(bits);
  }
  R.maxpairs = 1, R.maxrows = 1;
  for (auto [b, e] : parts) {
    RecGroup G{};
    G.row0 = brow0[b], G.nrows = brow0[e] - brow0[b];
    G.x0 = bx0[b], G.nx = bx0[e] - bx0[b];
    G.k0 = bk0[b], G.npath = bk0[e] - bk0[b];
    G.pair0 = row_pair[G.row0];
    G.npairs = row_pair[G.row0 + G.nrows] - G.pair0;
    R.maxpairs = std::max(R.maxpairs, G.npairs);
    R.maxrows = std::max(R.maxrows, G.nrows);
    for (int pp = G.pair0; pp < G.pair0 + G.npairs; ++pp) {
      const int xl = pi1[pp] - G.x0;
      if (xl < 0 || xl >= G.nx) {
        why = "a coupling record reads an x row outside its block";
        return false;
      }
      T[R.o_pxl + pp] = xl * kWave;
    }
    // rows: pair starts, then path-local index | last row of its path << 8
    G.rowtab = (int)T.size();
    for (int r = 0; r <= G.nrows; ++r) T.push_back(row_pair[G.row0 + r] - G.pair0);
    for (int k = G.k0; k < G.k0 + G.npath; ++k) {
      const int rows = 2 * L.paths[k].l3 + 1;
      for (int m = 0; m < rows; ++m) T.push_back((k - G.k0) | ((m == rows - 1) << 8));
    }
    // pairs by x row
    G.ttab = (int)T.size();
    {
      std::vector<std::vector<int>> by_x(G.nx);
      for (int pp = G.pair0; pp < G.pair0 + G.npairs; ++pp)
        by_x[pi1[pp] - G.x0].push_back((pp - G.pair0) | ((pi0[pp] - G.row0) << 16));
      int c = 0;
      for (int xl = 0; xl < G.nx; ++xl) T.push_back(c), c += (int)by_x[xl].size();
      T.push_back(c);
      for (auto& v : by_x)
        for (int ent : v) T.push_back(ent);
    }
    // records by harmonic index
    G.dytab = (int)T.size();
    {
      std::vector<std::vector<std::pair<int, int>>> by_y(L.d_sh);
      for (int r = prb[G.pair0]; r < prb[G.pair0 + G.npairs]; ++r) {
        const auto& c = p->recs[r];
        const float f = (float)c.v;
        int bits;
        std::memcpy(&bits, &f, 4);
        by_y[c.i2].push_back({(c.i1 - G.x0) | ((c.i0 - G.row0) << 8), bits});
      }
      int c = 0;
      for (int i = 0; i < L.d_sh; ++i) T.push_back(c), c += (int)by_y[i].size();
      T.push_back(c);
      for (auto& v : by_y)
        for (auto [ent, bits] : v) T.push_back(ent), T.push_back(bits);
    }
    R.groups.push_back(G);
  }
  R.nslab = (L.C + kWave - 1) / kWave;
  return true;
}

// Every index the kernels take from the tables, checked against the bounds
// of the arrays it addresses (the kernels trust the tables).
bool rec_validate(const e3_plan* p, const RecPlan& R, std::string& why) {
  const auto& L = p->lay;
  const std::vector<int>& T = R.tab;
  const int64_t nt = (int64_t)T.size(), nrec = (int64_t)p->recs.size();
  const int64_t npair = R.o_prb - R.o_pxl;
  auto in = [&](int64_t off, int64_t len) { return off >= 0 && len >= 0 && off + len <= nt; };
  auto fail = [&](const char* what) {
    why = std::string("record table check failed: ") + what;
    return false;
  };
  if (!in(R.o_pxl, npair) || !in(R.o_prb, npair + 1) || !in(R.o_ri2, nrec) || !in(R.o_rc, nrec))
    return fail("array offsets");
  for (int64_t i = 0; i < nrec; ++i)
    if (T[R.o_ri2 + i] < 0 || T[R.o_ri2 + i] >= L.d_sh) return fail("harmonic index");
  if (T[R.o_prb] != 0 || T[R.o_prb + npair] != nrec) return fail("record ranges");
  for (int64_t i = 0; i < npair; ++i)
    if (T[R.o_prb + i] > T[R.o_prb + i + 1]) return fail("record ranges");
  int rows = 0, xs = 0, ks = 0;
  for (const auto& G : R.groups) {
    if (G.row0 != rows || G.nrows < 0 || G.nrows > kRecRows || G.nrows > R.maxrows) return fail("group rows");
    if (G.x0 != xs || G.nx < 1 || G.nx > kRecX) return fail("group x rows");
    if (G.k0 != ks || G.npath < 0 || G.npath > kRecPaths) return fail("group paths");
    if (G.pair0 < 0 || G.npairs < 0 || G.pair0 + G.npairs > npair || G.npairs > R.maxpairs)
      return fail("group pairs");
    rows += G.nrows, xs += G.nx, ks += G.npath;
    for (int i = G.pair0; i < G.pair0 + G.npairs; ++i) {
      const int v = T[R.o_pxl + i];
      if (v % kWave != 0 || v < 0 || v / kWave >= G.nx) return fail("pair x row");
    }
    if (!in(G.rowtab, 2 * (int64_t)G.nrows + 1)) return fail("row table");
    if (T[G.rowtab] != 0 || T[G.rowtab + G.nrows] != G.npairs) return fail("row pair starts");
    for (int r = 0; r < G.nrows; ++r) {
      if (T[G.rowtab + r] > T[G.rowtab + r + 1]) return fail("row pair starts");
      const int info = T[G.rowtab + G.nrows + 1 + r];
      if ((info & 0xff) >= G.npath || (info >> 8) > 1) return fail("row path");
    }
    if (!in(G.ttab, (int64_t)G.nx + 1)) return fail("x table");
    const int nt_ent = T[G.ttab + G.nx];
    if (T[G.ttab] != 0 || !in(G.ttab + G.nx + 1, nt_ent)) return fail("x table entries");
    for (int xl = 0; xl < G.nx; ++xl)
      if (T[G.ttab + xl] > T[G.ttab + xl + 1]) return fail("x table starts");
    for (int u = 0; u < nt_ent; ++u) {
      const int ent = T[G.ttab + G.nx + 1 + u];
      if ((ent & 0xffff) >= G.npairs || (ent >> 16) >= G.nrows || ent < 0) return fail("x table entry");
    }
    if (!in(G.dytab, (int64_t)L.d_sh + 1)) return fail("harmonic table");
    const int ny = T[G.dytab + L.d_sh];
    if (T[G.dytab] != 0 || !in(G.dytab + L.d_sh + 1, 2 * (int64_t)ny)) return fail("harmonic table entries");
    for (int i = 0; i < L.d_sh; ++i)
      if (T[G.dytab + i] > T[G.dytab + i + 1]) return fail("harmonic table starts");
    for (int u = 0; u < ny; ++u) {
      const int ent = T[G.dytab + L.d_sh + 1 + 2 * u];
      if ((ent & 0xff) >= G.nx || (ent >> 8) >= G.nrows || ent < 0) return fail("harmonic table entry");
    }
  }
  if (rows != L.d_out || xs != L.d_in || ks != (int)L.paths.size()) return fail("group cover");
  return true;
}

size_t rec_lds_bytes(const RecPlan& R, bool bwd) {
  size_t f = kRecBatch * 16 + (size_t)kRecBatch * R.maxpairs + kRecX * kWave + kRecPaths * kWave;
  if (bwd) f += (size_t)R.maxrows * kWave;
  return f * sizeof(float);
}

}  // namespace

bool rec_ready(const e3_plan* p) { return p && p->rec && p->rec->dev; }

e3_status rec_create(e3_plan* p) {
  RecPlan R;
  std::string why;
  if (!rec_tables(p, R, why)) {
    g_last_error = "no compiled kernel variant for this layout, and the record path does not take it: " + why;
    return E3_ERR_UNSUPPORTED;
  }
  if (!rec_validate(p, R, why)) {
    g_last_error = why;
    return E3_ERR_UNSUPPORTED;
  }
  if (rec_lds_bytes(R, true) > 64 * 1024) {
    g_last_error = "the record path's LDS footprint exceeds 64 KiB for this layout";
    return E3_ERR_UNSUPPORTED;
  }
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || ndev <= 0) {
    (void)hipGetLastError();
    g_last_error = "no compiled kernel variant for this layout, and no device to hold the record path's tables";
    return E3_ERR_UNSUPPORTED;
  }
  const size_t gbytes = R.groups.size() * sizeof(RecGroup), tbytes = std::max<size_t>(4, R.tab.size() * 4);
  std::vector<char> host(gbytes + tbytes, 0);
  std::memcpy(host.data(), R.groups.data(), gbytes);
  if (!R.tab.empty()) std::memcpy(host.data() + gbytes, R.tab.data(), R.tab.size() * 4);
  E3_HIP(hipGetDevice(&R.device));
  char* d = nullptr;
  E3_HIP(hipMalloc(&d, host.size()));
  const hipError_t e = hipMemcpy(d, host.data(), host.size(), hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    g_last_error = std::string("record path tables upload: ") + hipGetErrorString(e);
    (void)hipFree(d);
    return E3_ERR_HIP;
  }
  R.dev = d;
  p->rec = new (std::nothrow) RecPlan(std::move(R));
  if (!p->rec) {
    (void)hipFree(d);
    return E3_ERR_ALLOC;
  }
  return E3_OK;
}

e3_status rec_check(const e3_plan* p) {
  if (p->composed) return E3_OK;
  if (!rec_ready(p)) {
    g_last_error = p->no_rec_reason;
    return E3_ERR_UNSUPPORTED;
  }
  int cur = -1;
  E3_HIP(hipGetDevice(&cur));
  if (cur != p->rec->device) {
    g_last_error = "the plan's record tables were uploaded to device " + std::to_string(p->rec->device) +
                   ", called with device " + std::to_string(cur) + " current";
    return E3_ERR_INVALID_ARG;
  }
  return E3_OK;
}

namespace {

RecArgs rec_args(const e3_plan* p, const e3_graph* g, int64_t rows) {
  const RecPlan& R = *p->rec;
  RecArgs a{};
  a.grp = reinterpret_cast<const RecGroup*>(R.dev);
  a.tab = reinterpret_cast<const int*>(R.dev + R.groups.size() * sizeof(RecGroup));
  a.o_pxl = R.o_pxl, a.o_prb = R.o_prb, a.o_ri2 = R.o_ri2, a.o_rc = R.o_rc;
  a.C = p->lay.C;
  a.nslab = R.nslab;
  a.ng = (int)R.groups.size();
  a.d_in = p->lay.d_in, a.d_out = p->lay.d_out, a.np = (int)p->lay.paths.size();
  a.maxpairs = R.maxpairs, a.maxrows = R.maxrows;
  if (g) {
    a.rowptr = g->rowptr_r, a.eid = g->eid_r, a.src = g->src_r, a.r2s = g->r2s;
    a.n_nodes = (int)g->n_nodes;
  } else {
    a.ident = 1;
    a.n_nodes = (int)rows;
  }
  a.chunk = (int)((a.n_nodes + kXcd - 1) / kXcd);
  return a;
}

int64_t rec_grid(const RecArgs& a) { return (int64_t)kXcd * a.chunk * a.ng * a.nslab; }

template <class K>
e3_status rec_launch(K kern, const RecArgs& a, size_t lds, const char* name, hipStream_t st) {
  const int64_t grid = rec_grid(a);
  if (grid > 0x7fffffff) {
    g_last_error = "the record path's grid exceeds 2^31 waves";
    return E3_ERR_UNSUPPORTED;
  }
  TimedLaunch t_(name, st);
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kWave), lds, st, a);
  E3_HIP(hipGetLastError());
  return E3_OK;
}

template <int L>
e3_status rec_fwd_l(const RecArgs& a, size_t lds, hipStream_t st) {
  return rec_launch(k_convr_fwd<L>, a, lds, "convr_fwd", st);
}
template <int L>
e3_status rec_bwd_l(const RecArgs& a, size_t lds, hipStream_t st) {
  return rec_launch(k_convr_bwd<L>, a, lds, "convr_bwd", st);
}

}  // namespace

// ------------------------------------------------------------ composed path
e3_status comp_create(e3_plan* p) {
  const auto& L = p->lay;
  const int C = L.C;
  if (C < 4 || C % 4 != 0 || C > kMaxChannels || L.lmax_out > 3) return E3_ERR_UNSUPPORTED;
  const int nb = (int)L.blocks.size();
  std::vector<e3_plan::KindBlock> kb;
  std::vector<std::pair<int, int>> pathless;
  int x_off = 0, k = 0, g0 = 0;
  for (int b = 0; b < nb; ++b) {
    const auto& B = L.blocks[b];
    if (B.l > 3) return E3_ERR_UNSUPPORTED;
    const int d1 = 2 * B.l + 1;
    const int k0 = k;
    while (k < (int)L.paths.size() && L.paths[k].xb == b) ++k;
    if (k == k0) {
      pathless.push_back({x_off, d1});
      x_off += d1;
      continue;
    }
    // the same block alone: its path list selects the kind
    e3b::Layout one;
    std::string err;
    const std::string irr = "1x" + std::to_string(B.l) + (B.p > 0 ? "e" : "o");
    if (!e3b::make_layout(irr, L.lmax_sh, L.lmax_out, L.natural, one, err)) return E3_ERR_UNSUPPORTED;
    if ((int)one.paths.size() != k - k0) return E3_ERR_UNSUPPORTED;
    for (int j = 0; j < k - k0; ++j) {
      const auto& a = L.paths[k0 + j];
      const auto& o = one.paths[j];
      if (a.l1 != o.l1 || a.l2 != o.l2 || a.l3 != o.l3 || a.x_off != x_off || a.out_off != L.paths[k0].out_off + o.out_off)
        return E3_ERR_UNSUPPORTED;
    }
    const std::string sig = e3b::path_signature(one);
    int kind = -1;
    for (int i = 0; i < kNumKinds; ++i)
      if (sig == kKinds[i]()->sig && one.d_sh == kKinds[i]()->d_sh) kind = i;
    if (kind < 0) return E3_ERR_UNSUPPORTED;
    const KindOps& K = *kKinds[kind]();
    if (K.d_in != d1 || K.np != k - k0 || K.d_out != one.d_out) return E3_ERR_UNSUPPORTED;
    kb.push_back({kind, x_off, k0, L.paths[k0].out_off, g0});
    g0 += K.nbg;
    x_off += d1;
  }
  if (x_off != L.d_in || k != (int)L.paths.size()) return E3_ERR_UNSUPPORTED;
  p->kblocks = std::move(kb);
  p->pathless = std::move(pathless);
  p->kng = g0;
  p->composed = true;
  p->cpl_f = C <= kWave ? 1 : E3_FWD_CPL;
  p->nslab_f = (C + kWave * p->cpl_f - 1) / (kWave * p->cpl_f);
  p->cpl_b = 1;
  p->nslab_b = (C + kWave - 1) / kWave;
  return E3_OK;
}

namespace {

KindCall comp_call(const e3_plan* p, int g0) {
  return KindCall{p->lay.d_in, (int)p->lay.paths.size(), p->lay.d_out, p->kng, g0};
}

e3_status comp_zero_rows(float* base, int64_t n, int64_t stride, int64_t off, int64_t len, hipStream_t st) {
  if (n == 0 || len == 0) return E3_OK;
  TimedLaunch t_("kind_zero_rows", st);
  hipLaunchKernelGGL(k_zero_rows, dim3(blocks_for(n * len, 256)), dim3(256), 0, st, base, n, stride, off, len);
  E3_HIP(hipGetLastError());
  return E3_OK;
}

Ws comp_ws(const e3_plan* p, const e3_graph* g) {
  Ws w{};
  w.t_bytes = align256((size_t)g->n_live * p->lay.d_in * p->lay.C * sizeof(float));
  w.dy_bytes = align256((size_t)g->n_live * p->kng * p->nslab_b * 16 * sizeof(float));
  return w;
}

template <int L>
e3_status launch_dvec(const float* vec, const float* DY, const int* eid, float* dvec, int64_t n, int nparts,
                      hipStream_t st) {
  hipLaunchKernelGGL(k_convr_dvec<L>, dim3(blocks_for(n, 256)), dim3(256), 0, st, vec, DY, eid, dvec, n, nparts);
  E3_HIP(hipGetLastError());
  return E3_OK;
}

// dvec / dy from the harmonic partials, zero rows of padding edges.
e3_status finish_bwd(const e3_plan* p, const e3_graph* g, int64_t n_live, const float* vec, const float* DY,
                     float* dvec, float* dy, float* ds, int nparts, int accum, hipStream_t st) {
  const int lsh = p->lay.lmax_sh, dsh = p->lay.d_sh;
  const int* eid = g ? g->eid_r : nullptr;
  if (n_live > 0 && dvec) {
    if (!g) return E3_ERR_INVALID_ARG;
    TimedLaunch t_("convr_dvec", st);
    e3_status s2;
    switch (lsh) {
      case 0: s2 = launch_dvec<0>(vec, DY, eid, dvec, n_live, nparts, st); break;
      case 1: s2 = launch_dvec<1>(vec, DY, eid, dvec, n_live, nparts, st); break;
      case 2: s2 = launch_dvec<2>(vec, DY, eid, dvec, n_live, nparts, st); break;
      default: s2 = launch_dvec<3>(vec, DY, eid, dvec, n_live, nparts, st); break;
    }
    if (s2 != E3_OK) return s2;
  }
  if (n_live > 0 && dy) {
    TimedLaunch t_("convr_dy", st);
    hipLaunchKernelGGL(k_convr_dy, dim3(blocks_for(n_live * dsh, 256)), dim3(256), 0, st, DY, eid, dy, n_live, dsh,
                       nparts, (accum & kAccDy) != 0);
    E3_HIP(hipGetLastError());
  }
  // padding edges: zero cotangents (left unchanged when accumulating)
  if (g && g->n_pad > 0) {
    float* z0 = (accum & kAccDs) ? nullptr : ds;
    float* z1 = dvec ? dvec : ((accum & kAccDy) ? nullptr : dy);
    const int64_t w1 = dvec ? 3 : dsh;
    if (z0 || z1) {
      TimedLaunch t_("conv_bwd_pad", st);
      hipLaunchKernelGGL(k_zero_pad, dim3((unsigned)g->n_pad), dim3(256), 0, st, g->eid_r + g->n_live, g->n_pad,
                         z0, (int64_t)p->lay.paths.size() * p->lay.C, z1, w1);
      E3_HIP(hipGetLastError());
    }
  }
  return E3_OK;
}

e3_status comp_fwd(const e3_plan* p, const e3_graph* g, int64_t rows, const float* x, const float* vec,
                   const float* y, const float* s, float* m, int accum, hipStream_t st) {
  const int64_t C = p->lay.C;
  for (const auto& b : p->kblocks) {
    const KindOps& K = *kKinds[b.kind]();
    const KindCall kc = comp_call(p, b.g0);
    e3_status r = g ? K.fwd(p, g, x + b.x_off * C, vec, y, s + b.k0 * C, m + b.o_off * C, accum, kc, st)
                    : K.tp(p, x + b.x_off * C, y, s + b.k0 * C, m + b.o_off * C, rows, kc, st);
    if (r != E3_OK) return r;
  }
  return E3_OK;
}

e3_status comp_bwd(const e3_plan* p, const e3_graph* g, int64_t rows, const float* x, const float* vec,
                   const float* y, const float* s, const float* dm, float* dx, float* dvec, float* dy, float* ds,
                   int accum, void* ws, hipStream_t st) {
  const int64_t C = p->lay.C, D_in = p->lay.d_in, P = (int64_t)p->lay.paths.size();
  const int nparts = p->kng * p->nslab_b;
  e3_status r;
  if (!g) {  // tensor product: dx and dw rows stored directly
    float* DY = reinterpret_cast<float*>(ws);
    for (const auto& b : p->kblocks) {
      const KindOps& K = *kKinds[b.kind]();
      if ((r = K.tpb(p, x + b.x_off * C, y, s + b.k0 * C, dm + b.o_off * C, dx + b.x_off * C, ds + b.k0 * C, DY,
                     rows, comp_call(p, b.g0), st)) != E3_OK)
        return r;
    }
    for (const auto& z : p->pathless)
      if ((r = comp_zero_rows(dx, rows, D_in * C, z.first * C, z.second * C, st)) != E3_OK) return r;
    return finish_bwd(p, nullptr, rows, nullptr, DY, nullptr, dy, nullptr, nparts, 0, st);
  }
  if (g->n_nodes == 0) return E3_OK;
  const Ws w = comp_ws(p, g);
  float* T = reinterpret_cast<float*>(ws);
  float* DY = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + w.t_bytes);
  for (const auto& b : p->kblocks) {
    const KindOps& K = *kKinds[b.kind]();
    const int64_t t_row = dx ? (int64_t)K.d_in * C * 4 : 0, ds_row = ds ? (int64_t)K.np * C * 4 : 0;
    if ((r = K.bwd(p, g, x + b.x_off * C, vec, y, s + b.k0 * C, dm + b.o_off * C, T + b.x_off * C, t_row, DY,
                   ds ? ds + b.k0 * C : DY, ds_row, (accum & kAccDs) != 0, comp_call(p, b.g0), st)) != E3_OK)
      return r;
  }
  if (dx) {
    for (const auto& z : p->pathless)
      if ((r = comp_zero_rows(T, g->n_live, D_in * C, z.first * C, z.second * C, st)) != E3_OK) return r;
    TimedLaunch t_("conv_bwd_dx", st);
    const int flat4 = (int)(D_in * C / 4);
    const int nsl = (flat4 + kWave * kDxVec - 1) / (kWave * kDxVec);
    const int chunk = (int)((g->n_nodes + kXcd - 1) / kXcd);
    hipLaunchKernelGGL(k_conv_bwd_dx, dim3((unsigned)(kXcd * chunk * nsl)), dim3(kWave), 0, st, T, dx, g->rowptr_s,
                       (int)g->n_nodes, chunk, flat4, nsl, (accum & kAccDx) != 0);
    E3_HIP(hipGetLastError());
  }
  (void)P;
  return finish_bwd(p, g, g->n_live, vec, DY, dvec, dy, ds, nparts, accum, st);
}

}  // namespace

Ws rec_ws(const e3_plan* p, const e3_graph* g) {
  if (p->composed) return comp_ws(p, g);
  Ws w{};
  const RecPlan& R = *p->rec;
  w.t_bytes = align256((size_t)g->n_live * p->lay.d_in * p->lay.C * sizeof(float));
  w.dy_bytes = align256((size_t)g->n_live * R.groups.size() * R.nslab * 16 * sizeof(float));
  return w;
}

size_t rec_tp_ws(const e3_plan* p, int64_t rows) {
  if (p->composed) return align256((size_t)rows * p->kng * p->nslab_b * 16 * sizeof(float));
  const RecPlan& R = *p->rec;
  return align256((size_t)rows * R.groups.size() * R.nslab * 16 * sizeof(float));
}

e3_status rec_fwd(const e3_plan* p, const e3_graph* g, int64_t rows, const float* x, const float* vec,
                  const float* y, const float* s, float* m, int accum, hipStream_t st) {
  const int64_t n = g ? g->n_nodes : rows;
  if (n == 0) return E3_OK;
  if (n > 0x7fffffff) return E3_ERR_UNSUPPORTED;
  if (p->composed) return comp_fwd(p, g, rows, x, vec, y, s, m, accum, st);
  RecArgs a = rec_args(p, g, rows);
  a.x = x, a.vec = vec, a.y = y, a.s = s, a.m = m, a.accum = accum;
  const size_t lds = rec_lds_bytes(*p->rec, false);
  switch (p->lay.lmax_sh) {
    case 0: return rec_fwd_l<0>(a, lds, st);
    case 1: return rec_fwd_l<1>(a, lds, st);
    case 2: return rec_fwd_l<2>(a, lds, st);
    default: return rec_fwd_l<3>(a, lds, st);
  }
}

e3_status rec_bwd(const e3_plan* p, const e3_graph* g, int64_t rows, const float* x, const float* vec,
                  const float* y, const float* s, const float* dm, float* dx, float* dvec, float* dy, float* ds,
                  int accum, void* ws, hipStream_t st) {
  const int64_t n = g ? g->n_nodes : rows;
  if (n == 0) return E3_OK;
  if (n > 0x7fffffff) return E3_ERR_UNSUPPORTED;
  if (p->composed) return comp_bwd(p, g, rows, x, vec, y, s, dm, dx, dvec, dy, ds, accum, ws, st);
  const RecPlan& R = *p->rec;
  const int64_t n_live = g ? g->n_live : rows;
  const int lsh = p->lay.lmax_sh, dsh = p->lay.d_sh, C = p->lay.C;
  const int nparts = (int)R.groups.size() * R.nslab;
  RecArgs a = rec_args(p, g, rows);
  a.x = x, a.vec = vec, a.y = y, a.s = s, a.dm = dm, a.accum = (accum & kAccDs) != 0;
  if (g) {
    const Ws w = rec_ws(p, g);
    a.T = reinterpret_cast<float*>(ws);
    a.DY = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + w.t_bytes);
  } else {  // one edge per row: the x-cotangent partial of row r is dx[r]
    a.T = dx;
    a.DY = reinterpret_cast<float*>(ws);
  }
  a.ds = ds ? ds : a.DY;
  a.ds_row = ds ? (int64_t)a.np * C * 4 : 0;
  a.t_row = dx ? (int64_t)p->lay.d_in * C * 4 : 0;
  if (!g && dx && (accum & kAccDx)) return E3_ERR_UNSUPPORTED;
  if (n_live > 0) {
    const size_t lds = rec_lds_bytes(R, true);
    e3_status s2;
    switch (lsh) {
      case 0: s2 = rec_bwd_l<0>(a, lds, st); break;
      case 1: s2 = rec_bwd_l<1>(a, lds, st); break;
      case 2: s2 = rec_bwd_l<2>(a, lds, st); break;
      default: s2 = rec_bwd_l<3>(a, lds, st); break;
    }
    if (s2 != E3_OK) return s2;
  }
  if (g && dx) {
    TimedLaunch t_("conv_bwd_dx", st);
    const int flat4 = p->lay.d_in * C / 4;
    const int nsl = (flat4 + kWave * kDxVec - 1) / (kWave * kDxVec);
    hipLaunchKernelGGL(k_conv_bwd_dx, dim3((unsigned)(kXcd * a.chunk * nsl)), dim3(kWave), 0, st, a.T, dx,
                       g->rowptr_s, a.n_nodes, a.chunk, flat4, nsl, (accum & kAccDx) != 0);
    E3_HIP(hipGetLastError());
  }
  const int* eid = g ? g->eid_r : nullptr;
  if (n_live > 0 && dvec) {
    if (!g) return E3_ERR_INVALID_ARG;
    TimedLaunch t_("convr_dvec", st);
    const dim3 gr(blocks_for(n_live, 256)), bl(256);
    switch (lsh) {
      case 0: hipLaunchKernelGGL(k_convr_dvec<0>, gr, bl, 0, st, vec, a.DY, eid, dvec, n_live, nparts); break;
      case 1: hipLaunchKernelGGL(k_convr_dvec<1>, gr, bl, 0, st, vec, a.DY, eid, dvec, n_live, nparts); break;
      case 2: hipLaunchKernelGGL(k_convr_dvec<2>, gr, bl, 0, st, vec, a.DY, eid, dvec, n_live, nparts); break;
      default: hipLaunchKernelGGL(k_convr_dvec<3>, gr, bl, 0, st, vec, a.DY, eid, dvec, n_live, nparts); break;
    }
    E3_HIP(hipGetLastError());
  }
  if (n_live > 0 && dy) {
    TimedLaunch t_("convr_dy", st);
    hipLaunchKernelGGL(k_convr_dy, dim3(blocks_for(n_live * dsh, 256)), dim3(256), 0, st, a.DY, eid, dy, n_live,
                       dsh, nparts, (accum & kAccDy) != 0);
    E3_HIP(hipGetLastError());
  }
  // padding edges: zero cotangents (left unchanged when accumulating)
  if (g && g->n_pad > 0) {
    float* z0 = (accum & kAccDs) ? nullptr : ds;
    float* z1 = dvec ? dvec : ((accum & kAccDy) ? nullptr : dy);
    const int64_t w1 = dvec ? 3 : dsh;
    if (z0 || z1) {
      TimedLaunch t_("conv_bwd_pad", st);
      hipLaunchKernelGGL(k_zero_pad, dim3((unsigned)g->n_pad), dim3(256), 0, st, g->eid_r + g->n_live, g->n_pad,
                         z0, (int64_t)a.np * C, z1, w1);
      E3_HIP(hipGetLastError());
    }
  }
  return E3_OK;
}

// ------------------------------------------------------------ composed path, float64
namespace {
int nslab_c64(const e3_plan* p) { return (p->lay.C + kWave - 1) / kWave; }

template <int L>
e3_status launch_dvec64(const double* vec, const double* DY, const int* eid, double* dvec, int64_t n, int nparts,
                        hipStream_t st) {
  hipLaunchKernelGGL(k_convr_dvec64<L>, dim3(blocks_for(n, 256)), dim3(256), 0, st, vec, DY, eid, dvec, n, nparts);
  E3_HIP(hipGetLastError());
  return E3_OK;
}
}  // namespace

Ws comp_ws64(const e3_plan* p, const e3_graph* g) {
  Ws w{};
  w.t_bytes = align256((size_t)g->n_live * p->lay.d_in * p->lay.C * sizeof(double));
  w.dy_bytes = align256((size_t)g->n_live * p->kng * nslab_c64(p) * 16 * sizeof(double));
  return w;
}

size_t comp_tp_ws64(const e3_plan* p, int64_t rows) {
  return align256((size_t)rows * p->kng * nslab_c64(p) * 16 * sizeof(double));
}

e3_status comp_fwd64(const e3_plan* p, const e3_graph* g, const double* x, const double* vec, const double* s,
                     double* m, hipStream_t st) {
  if (g->n_nodes == 0) return E3_OK;
  const int64_t C = p->lay.C;
  for (const auto& b : p->kblocks) {
    const KindOps& K = *kKinds[b.kind]();
    e3_status r = K.fwd64(p, g, x + b.x_off * C, vec, s + b.k0 * C, m + b.o_off * C, comp_call(p, b.g0), st);
    if (r != E3_OK) return r;
  }
  return E3_OK;
}

e3_status comp_bwd64(const e3_plan* p, const e3_graph* g, const double* x, const double* vec, const double* s,
                     const double* dm, double* dx, double* dvec, double* ds, void* ws, hipStream_t st) {
  if (g->n_nodes == 0) return E3_OK;
  const int64_t C = p->lay.C, D_in = p->lay.d_in, P = (int64_t)p->lay.paths.size();
  const int nsl = nslab_c64(p), nparts = p->kng * nsl;
  const Ws w = comp_ws64(p, g);
  double* T = reinterpret_cast<double*>(ws);
  double* DY = reinterpret_cast<double*>(reinterpret_cast<char*>(ws) + w.t_bytes);
  e3_status r;
  for (const auto& b : p->kblocks) {
    const KindOps& K = *kKinds[b.kind]();
    if ((r = K.bwd64(p, g, x + b.x_off * C, vec, s + b.k0 * C, dm + b.o_off * C, T + b.x_off * C, DY,
                     ds + b.k0 * C, comp_call(p, b.g0), st)) != E3_OK)
      return r;
  }
  // zero partial rows of blocks without paths, as pairs of 32-bit zeros
  for (const auto& z : p->pathless)
    if ((r = comp_zero_rows(reinterpret_cast<float*>(T), g->n_live, 2 * D_in * C, 2 * z.first * C, 2 * z.second * C,
                            st)) != E3_OK)
      return r;
  {
    TimedLaunch t_("conv_bwd_dx_f64", st);
    hipLaunchKernelGGL(k_conv_bwd_dx64, dim3((unsigned)(g->n_nodes * nsl)), dim3(kWave), 0, st, T, dx, g->rowptr_s,
                       (int)g->n_nodes, (int)D_in, (int)C, nsl);
    E3_HIP(hipGetLastError());
  }
  if (g->n_live > 0) {
    TimedLaunch t_("convr_dvec_f64", st);
    switch (p->lay.lmax_sh) {
      case 0: r = launch_dvec64<0>(vec, DY, g->eid_r, dvec, g->n_live, nparts, st); break;
      case 1: r = launch_dvec64<1>(vec, DY, g->eid_r, dvec, g->n_live, nparts, st); break;
      case 2: r = launch_dvec64<2>(vec, DY, g->eid_r, dvec, g->n_live, nparts, st); break;
      default: r = launch_dvec64<3>(vec, DY, g->eid_r, dvec, g->n_live, nparts, st); break;
    }
    if (r != E3_OK) return r;
  }
  if (g->n_pad > 0) {  // padding edges: zero ds and dvec rows (as pairs of 32-bit zeros)
    TimedLaunch t_("conv_bwd_pad", st);
    hipLaunchKernelGGL(k_zero_pad, dim3((unsigned)g->n_pad), dim3(256), 0, st, g->eid_r + g->n_live, g->n_pad,
                       reinterpret_cast<float*>(ds), (int64_t)2 * P * C, reinterpret_cast<float*>(dvec), (int64_t)6);
    E3_HIP(hipGetLastError());
  }
  return E3_OK;
}

e3_status comp_tp64(const e3_plan* p, const double* x, const double* y, const double* w, double* z, int64_t rows,
                    hipStream_t st) {
  const int64_t C = p->lay.C;
  for (const auto& b : p->kblocks) {
    const KindOps& K = *kKinds[b.kind]();
    e3_status r = K.tp64(p, x + b.x_off * C, y, w + b.k0 * C, z + b.o_off * C, rows, comp_call(p, b.g0), st);
    if (r != E3_OK) return r;
  }
  return E3_OK;
}

e3_status comp_tpb64(const e3_plan* p, const double* x, const double* y, const double* w, const double* dz,
                     double* dx, double* dy, double* dw, void* ws, int64_t rows, hipStream_t st) {
  const int64_t C = p->lay.C, D_in = p->lay.d_in;
  const int nparts = p->kng * nslab_c64(p);
  double* DY = reinterpret_cast<double*>(ws);
  e3_status r;
  for (const auto& b : p->kblocks) {
    const KindOps& K = *kKinds[b.kind]();
    if ((r = K.tpb64(p, x + b.x_off * C, y, w + b.k0 * C, dz + b.o_off * C, dx + b.x_off * C, dw + b.k0 * C, DY,
                     rows, comp_call(p, b.g0), st)) != E3_OK)
      return r;
  }
  for (const auto& z : p->pathless)
    if ((r = comp_zero_rows(reinterpret_cast<float*>(dx), rows, 2 * D_in * C, 2 * z.first * C, 2 * z.second * C,
                            st)) != E3_OK)
      return r;
  TimedLaunch t_("convr_dy_f64", st);
  hipLaunchKernelGGL(k_convr_dy64, dim3(blocks_for(rows * p->lay.d_sh, 256)), dim3(256), 0, st, DY,
                     (const int*)nullptr, dy, rows, p->lay.d_sh, nparts);
  E3_HIP(hipGetLastError());
  return E3_OK;
}

// ------------------------------------------------------------ composed path, fused radial weights
RadWs comp_rad_ws(const e3_plan* p, const e3_graph* g, int K) {
  return rad_ws_of(p, g, K, (int)p->lay.paths.size(), comp_ws(p, g));
}

e3_status comp_fwd_rad(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* h,
                       const float* W, int K, float* m, hipStream_t st) {
  if (g->n_nodes == 0) return E3_OK;
  const int64_t C = p->lay.C;
  for (const auto& b : p->kblocks) {
    const KindOps& Kd = *kKinds[b.kind]();
    e3_status r = Kd.rfwd(p, g, x + b.x_off * C, vec, h, W + b.k0 * C, K, m + b.o_off * C, comp_call(p, b.g0), st);
    if (r != E3_OK) return r;
  }
  return E3_OK;
}

e3_status comp_bwd_rad(const e3_plan* p, const e3_graph* g, const float* x, const float* vec, const float* h,
                       const float* W, int K, const float* dm, float* dx, float* dvec, float* dh, float* dW,
                       void* ws, hipStream_t st) {
  const int64_t C = p->lay.C, D_in = p->lay.d_in;
  const RadWs w = comp_rad_ws(p, g, K);
  char* base = reinterpret_cast<char*>(ws);
  float* T = reinterpret_cast<float*>(base);
  float* DY = reinterpret_cast<float*>(base + w.t);
  float* DS = reinterpret_cast<float*>(base + w.t + w.dy);
  float* dWp = reinterpret_cast<float*>(base + w.t + w.dy + w.ds);
  float* DHp = reinterpret_cast<float*>(base + w.t + w.dy + w.ds + w.dwp);
  const int nparts = p->kng * p->nslab_b;
  e3_status r;
  for (const auto& b : p->kblocks) {
    const KindOps& Kd = *kKinds[b.kind]();
    if ((r = Kd.rbwd(p, g, x + b.x_off * C, vec, h, W + b.k0 * C, K, dm + b.o_off * C, T + b.x_off * C, DY,
                     DS + b.k0 * C, comp_call(p, b.g0), st)) != E3_OK)
      return r;
  }
  if (g->n_nodes > 0) {
    for (const auto& z : p->pathless)
      if ((r = comp_zero_rows(T, g->n_live, D_in * C, z.first * C, z.second * C, st)) != E3_OK) return r;
    TimedLaunch t_("conv_bwd_dx", st);
    const int flat4 = (int)(D_in * C / 4);
    const int nsl = (flat4 + kWave * kDxVec - 1) / (kWave * kDxVec);
    const int chunk = (int)((g->n_nodes + kXcd - 1) / kXcd);
    hipLaunchKernelGGL(k_conv_bwd_dx, dim3((unsigned)(kXcd * chunk * nsl)), dim3(kWave), 0, st, T, dx, g->rowptr_s,
                       (int)g->n_nodes, chunk, flat4, nsl, 0);
    E3_HIP(hipGetLastError());
  }
  if (g->n_live > 0) {
    if ((r = finish_bwd(p, g, g->n_live, vec, DY, dvec, nullptr, nullptr, nparts, 0, st)) != E3_OK) return r;
    if (g->n_pad > 0) {
      // the ds rows of padding edges enter the gradient sums: clear them
      TimedLaunch t_("rad_pad_ds", st);
      hipLaunchKernelGGL(k_zero_pad, dim3((unsigned)g->n_pad), dim3(256), 0, st, g->eid_r + g->n_live, g->n_pad, DS,
                         (int64_t)w.pc4 * 4, dvec, (int64_t)3);
      E3_HIP(hipGetLastError());
    }
    const int64_t E = g->n_edges;
    {
      TimedLaunch t_("rad_grad", st);
      const dim3 grid((unsigned)((int64_t)w.nchunk * w.nsl4));
      if (K <= 8)
        hipLaunchKernelGGL(k_rad_grad<2>, grid, dim3(kWave), 0, st, DS, h, W, dWp, DHp, E, w.pc4, K, w.nsl4,
                           w.rows_per);
      else
        hipLaunchKernelGGL(k_rad_grad<4>, grid, dim3(kWave), 0, st, DS, h, W, dWp, DHp, E, w.pc4, K, w.nsl4,
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

// ------------------------------------------------------------ composed path, double backward
e3_status comp_bwd2(const e3_plan* p, const e3_graph* g, const float* x, const float* y, const float* s,
                    const float* dm, const float* ddx, const float* ddy, const float* dds, float* gx, float* gy,
                    float* gs, float* gdm, void* ws, hipStream_t st) {
  if (g->n_nodes == 0) return E3_OK;
  const int64_t C = p->lay.C, D_in = p->lay.d_in;
  e3_status r;
  // gdm = conv(ddx, y, s) + conv(x, ddy, s) + conv(x, y, dds): one sweep per block
  for (const auto& b : p->kblocks) {
    const KindOps& K = *kKinds[b.kind]();
    if ((r = K.fwd3(p, g, x + b.x_off * C, ddx + b.x_off * C, y, ddy, s + b.k0 * C, dds + b.k0 * C,
                    gdm + b.o_off * C, comp_call(p, b.g0), st)) != E3_OK)
      return r;
  }
  // gx, gy, gs: the three backward terms in one sweep per block, then the
  // shared sender-order sum and harmonic sum
  const Ws w = comp_ws(p, g);
  float* T = reinterpret_cast<float*>(ws);
  float* DY = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + w.t_bytes);
  for (const auto& b : p->kblocks) {
    const KindOps& K = *kKinds[b.kind]();
    if ((r = K.bwd3(p, g, x + b.x_off * C, ddx + b.x_off * C, y, ddy, s + b.k0 * C, dds + b.k0 * C,
                    dm + b.o_off * C, T + b.x_off * C, DY, gs + b.k0 * C, comp_call(p, b.g0), st)) != E3_OK)
      return r;
  }
  for (const auto& z : p->pathless)
    if ((r = comp_zero_rows(T, g->n_live, D_in * C, z.first * C, z.second * C, st)) != E3_OK) return r;
  {
    TimedLaunch t_("conv_bwd_dx", st);
    const int flat4 = (int)(D_in * C / 4);
    const int nsl = (flat4 + kWave * kDxVec - 1) / (kWave * kDxVec);
    const int chunk = (int)((g->n_nodes + kXcd - 1) / kXcd);
    hipLaunchKernelGGL(k_conv_bwd_dx, dim3((unsigned)(kXcd * chunk * nsl)), dim3(kWave), 0, st, T, gx, g->rowptr_s,
                       (int)g->n_nodes, chunk, flat4, nsl, 0);
    E3_HIP(hipGetLastError());
  }
  return finish_bwd(p, g, g->n_live, nullptr, DY, nullptr, gy, gs, p->kng * p->nslab_b, 0, st);
}
