// Neighbour list, reverse-edge map, edge geometry and the radial basis.
//
// Paper Sec. "MatRIS": the graph generation module repeats a structure
// periodically and connects atoms closer than the cutoff; the embedding
// module turns distances into edge features.  The inclusion rule (an fp32
// expression with a fixed operation order and no fused multiply-add), the
// canonical (i, j, n) order and the basis are the readings documented with
// janus_build_edges and in the design notes.
#include <cmath>

#include "internal.h"
#include "kernels.h"

namespace janus {

// Image half-widths m_k = floor(r_cut / L_k) + 1 of a diagonal cell.
__device__ __forceinline__ void image_range(const float* L, float rc, int& mx, int& my, int& mz) {
  mx = (int)floor((double)rc / (double)L[0]) + 1;
  my = (int)floor((double)rc / (double)L[4]) + 1;
  mz = (int)floor((double)rc / (double)L[8]) + 1;
}

__global__ void validate_struct_kernel(const int* __restrict__ offsets, int S, int N, const float* __restrict__ cell,
                                       float rc, int* __restrict__ flag) {
  int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s > S) return;
  int bad = 0;
  if (s == 0 && offsets[0] != 0) bad |= 1;
  if (s == S && offsets[S] != N) bad |= 1;
  if (s < S) {
    if (offsets[s] > offsets[s + 1]) bad |= 1;
    if (rc > 0.f) {
      const float* L = cell + 9 * s;
      if (L[1] != 0.f || L[2] != 0.f || L[3] != 0.f || L[5] != 0.f || L[6] != 0.f || L[7] != 0.f) bad |= 2;
      if (!(L[0] > 0.f) || !(L[4] > 0.f) || !(L[8] > 0.f)) bad |= 2;
      // image shifts are stored as int8 and the candidate count must stay small
      else if ((double)rc / L[0] > 60.0 || (double)rc / L[4] > 60.0 || (double)rc / L[8] > 60.0) bad |= 2;
    }
  }
  if (bad) atomicOr(flag, bad);
}

// sid[a] = structure of atom a (clamped so that bad offsets cannot write out of range).
__global__ void atom_struct_kernel(const int* __restrict__ offsets, int S, int N, int* __restrict__ sid) {
  int s = blockIdx.x;
  if (s >= S) return;
  int a0 = max(0, min(N, offsets[s])), a1 = max(0, min(N, offsets[s + 1]));
  for (int a = a0 + threadIdx.x; a < a1; a += blockDim.x) sid[a] = s;
}

// The pinned inclusion test of the pair (i, image (ix, iy, iz) of j): every
// operation rounded to fp32 separately, in the documented order.
__device__ __forceinline__ void image_shift(const float* L, int ix, int iy, int iz, float& sx, float& sy,
                                            float& sz) {
  const float fx = (float)ix, fy = (float)iy, fz = (float)iz;
  sx = __fadd_rn(__fadd_rn(__fmul_rn(fx, L[0]), __fmul_rn(fy, L[3])), __fmul_rn(fz, L[6]));
  sy = __fadd_rn(__fadd_rn(__fmul_rn(fx, L[1]), __fmul_rn(fy, L[4])), __fmul_rn(fz, L[7]));
  sz = __fadd_rn(__fadd_rn(__fmul_rn(fx, L[2]), __fmul_rn(fy, L[5])), __fmul_rn(fz, L[8]));
}
__device__ __forceinline__ bool pair_kept(const float* __restrict__ pos, int i, int j, float xi, float yi, float zi,
                                          float sx, float sy, float sz, bool zero_image, float rc2) {
  const float dx = __fadd_rn(__fsub_rn(pos[3 * j], xi), sx);
  const float dy = __fadd_rn(__fsub_rn(pos[3 * j + 1], yi), sy);
  const float dz = __fadd_rn(__fsub_rn(pos[3 * j + 2], zi), sz);
  const float r2 = __fadd_rn(__fadd_rn(__fmul_rn(dx, dx), __fmul_rn(dy, dy)), __fmul_rn(dz, dz));
  return (r2 < rc2) && !(j == i && zero_image);
}

// Cell list of one structure: the bounding box of its atoms cut into nb[k]
// bins per dimension, each at least r_cut wide, at most n_s bins in all.
struct CellGrid {
  double lo[3];       // lower corner of the box
  double hi[3];       // upper corner
  double inv_w[3];    // bins per unit length (0 for a single bin)
  double margin[3];   // widening of every searched range, far above fp32 rounding
  int nb[3];
  int use;            // 1: the centres of this structure go through the cell-list kernels
};

// Per-centre capacity of the cell-list write pass (sort keys in LDS); a centre
// with more neighbours is written by the all-pairs kernel instead.
constexpr int kCellCap = 512;

// One wave per centre atom; candidates (j, image) are tested 64 at a time in
// canonical order and compacted with a ballot, so the output order is exact.
// Centres of structures that use the cell list are skipped (the write pass
// takes those whose neighbours exceed kCellCap).
template <bool WRITE>
__global__ void nl_kernel(const float* __restrict__ pos, const float* __restrict__ cell,
                          const int* __restrict__ offsets, const int* __restrict__ sid, float rc, int N,
                          int* __restrict__ count, const int* __restrict__ rowptr, int* __restrict__ ei,
                          int* __restrict__ ej, int8_t* __restrict__ shift, const CellGrid* __restrict__ grid) {
  const int i = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  if (i >= N) return;
  const int s = sid[i];
  if (grid[s].use && (!WRITE || count[i] <= kCellCap)) return;
  const int a = offsets[s], n = offsets[s + 1] - a;
  const float* L = cell + 9 * s;
  int mx, my, mz;
  image_range(L, rc, mx, my, mz);
  const int ny = 2 * my + 1, nz = 2 * mz + 1;
  const int nimg = (2 * mx + 1) * ny * nz;
  const float xi = pos[3 * i], yi = pos[3 * i + 1], zi = pos[3 * i + 2];
  const float rc2 = __fmul_rn(rc, rc);
  const long long ncand = (long long)n * nimg;
  const int base = WRITE ? rowptr[i] : 0;
  int cnt = 0;
  for (long long c0 = 0; c0 < ncand; c0 += 64) {
    const long long c = c0 + lane;
    bool keep = false;
    int j = 0, ix = 0, iy = 0, iz = 0;
    if (c < ncand) {
      j = a + (int)(c / nimg);
      const int im = (int)(c % nimg);
      ix = im / (ny * nz) - mx;
      iy = (im / nz) % ny - my;
      iz = im % nz - mz;
      float sx, sy, sz;
      image_shift(L, ix, iy, iz, sx, sy, sz);
      keep = pair_kept(pos, i, j, xi, yi, zi, sx, sy, sz, ix == 0 && iy == 0 && iz == 0, rc2);
    }
    const unsigned long long m = __ballot(keep);
    if (WRITE && keep) {
      const int p = base + cnt + __popcll(m & ((1ull << lane) - 1ull));
      ei[p] = i;
      ej[p] = j;
      shift[3 * p] = (int8_t)ix;
      shift[3 * p + 1] = (int8_t)iy;
      shift[3 * p + 2] = (int8_t)iz;
    }
    cnt += __popcll(m);
  }
  if (!WRITE && lane == 0) count[i] = cnt;
}

// ------------------------------------------------------------------ cell list
// A structure uses the cell list when mode says so (1: every structure, 2:
// none) or, in mode 0, when its all-pairs candidate count n_s * n_images is at
// least kCellMinCand and its box holds at least 27 bins.  Bins are built per
// structure from the atoms' own bounding box (positions need not be wrapped);
// a centre then tests, for every image n, only the atoms of the bins that the
// ball of radius r_cut around X_i - s(n) reaches, with the same fp32 test, and
// its kept (j, n) are sorted into the canonical order in LDS: the list is
// bitwise the all-pairs one.
constexpr long long kCellMinCand = 32768;

// One workgroup per structure: bounding box, bins, use flag; nbins[s] = bins used.
__global__ void cell_grid_kernel(const float* __restrict__ pos, const float* __restrict__ cell,
                                 const int* __restrict__ offsets, int S, float rc, int mode,
                                 CellGrid* __restrict__ grid, int* __restrict__ nbins) {
  __shared__ float red[6][256];
  const int s = blockIdx.x;
  if (s >= S) return;
  const int a = offsets[s], n = offsets[s + 1] - a;
  float lo[3] = {INFINITY, INFINITY, INFINITY}, hi[3] = {-INFINITY, -INFINITY, -INFINITY};
  for (int t = threadIdx.x; t < n; t += blockDim.x)
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      const float v = pos[3 * (a + t) + k];
      lo[k] = fminf(lo[k], v);
      hi[k] = fmaxf(hi[k], v);
    }
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    red[k][threadIdx.x] = lo[k];
    red[3 + k][threadIdx.x] = hi[k];
  }
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o)
#pragma unroll
      for (int k = 0; k < 3; ++k) {
        red[k][threadIdx.x] = fminf(red[k][threadIdx.x], red[k][threadIdx.x + o]);
        red[3 + k][threadIdx.x] = fmaxf(red[3 + k][threadIdx.x], red[3 + k][threadIdx.x + o]);
      }
    __syncthreads();
  }
  if (threadIdx.x != 0) return;
  CellGrid g;
  const float* L = cell + 9 * s;
  int m[3];
  image_range(L, rc, m[0], m[1], m[2]);
  long long bins = 1;
  for (int k = 0; k < 3; ++k) {
    const double l = n > 0 ? (double)red[k][0] : 0.0, h = n > 0 ? (double)red[3 + k][0] : 0.0;
    const double ext = h - l;
    int nb = (int)fmin(64.0, floor(ext / (double)rc));
    g.nb[k] = nb < 1 ? 1 : nb;
    g.lo[k] = l;
    g.hi[k] = h;
    g.margin[k] = 1e-4 * (fabs(l) + fabs(h) + (m[k] + 1.0) * (double)L[4 * k] + (double)rc);
  }
  // at most n_s bins: halve the widest dimension until the product fits
  while ((long long)g.nb[0] * g.nb[1] * g.nb[2] > (n > 1 ? n : 1)) {
    int k = 0;
    if (g.nb[1] > g.nb[k]) k = 1;
    if (g.nb[2] > g.nb[k]) k = 2;
    g.nb[k] = (g.nb[k] + 1) / 2;
  }
  for (int k = 0; k < 3; ++k) {
    const double ext = n > 0 ? (double)red[3 + k][0] - (double)red[k][0] : 0.0;
    g.inv_w[k] = (g.nb[k] > 1 && ext > 0.0) ? g.nb[k] / ext : 0.0;
  }
  bins = (long long)g.nb[0] * g.nb[1] * g.nb[2];
  const long long nimg = (long long)(2 * m[0] + 1) * (2 * m[1] + 1) * (2 * m[2] + 1);
  int use = 0;
  if (n > 0) use = mode == 1 ? 1 : mode == 2 ? 0 : ((long long)n * nimg >= kCellMinCand && bins >= 27);
  g.use = use;
  grid[s] = g;
  nbins[s] = use ? (int)bins : 0;
}

__device__ __forceinline__ int cell_coord(double x, const CellGrid& g, int k) {
  const double f = floor((x - g.lo[k]) * g.inv_w[k]);
  return f < 0.0 ? 0 : f > g.nb[k] - 1 ? g.nb[k] - 1 : (int)f;
}

// bin of every atom of a cell-list structure, and the atom count of every bin
__global__ void cell_bin_kernel(const float* __restrict__ pos, const int* __restrict__ sid,
                                const CellGrid* __restrict__ grid, const int* __restrict__ bin_off, int N,
                                int* __restrict__ abin, int* __restrict__ bcount) {
  const int at = blockIdx.x * blockDim.x + threadIdx.x;
  if (at >= N) return;
  const int s = sid[at];
  const CellGrid& g = grid[s];
  if (!g.use) return;
  const int bx = cell_coord(pos[3 * at], g, 0), by = cell_coord(pos[3 * at + 1], g, 1),
            bz = cell_coord(pos[3 * at + 2], g, 2);
  const int b = bin_off[s] + (bx * g.nb[1] + by) * g.nb[2] + bz;
  abin[at] = b;
  atomicAdd(bcount + b, 1);
}

// atoms listed by bin (any order inside a bin: the write pass sorts)
__global__ void cell_fill_kernel(const int* __restrict__ sid, const CellGrid* __restrict__ grid,
                                 const int* __restrict__ abin, const int* __restrict__ bstart, int N,
                                 int* __restrict__ bfill, int* __restrict__ batoms) {
  const int at = blockIdx.x * blockDim.x + threadIdx.x;
  if (at >= N) return;
  if (!grid[sid[at]].use) return;
  const int b = abin[at];
  batoms[bstart[b] + atomicAdd(bfill + b, 1)] = at;
}

__device__ __forceinline__ void cell_wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One wave per centre of a cell-list structure: count (WRITE = false) or
// collect, sort by (j, image) and write (WRITE = true, at most kCellCap).
template <bool WRITE>
__global__ __launch_bounds__(256) void nl_cell_kernel(
    const float* __restrict__ pos, const float* __restrict__ cell, const int* __restrict__ offsets,
    const int* __restrict__ sid, float rc, int N, const CellGrid* __restrict__ grid, const int* __restrict__ bin_off,
    const int* __restrict__ bstart, const int* __restrict__ batoms, int* __restrict__ count,
    const int* __restrict__ rowptr, int* __restrict__ ei, int* __restrict__ ej, int8_t* __restrict__ shift) {
  __shared__ unsigned long long keys_all[4][kCellCap];
  const int i = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  if (i >= N) return;
  const int s = sid[i];
  const CellGrid g = grid[s];
  if (!g.use) return;
  if (WRITE && count[i] > kCellCap) return;
  unsigned long long* keys = keys_all[threadIdx.x >> 6];
  const int a = offsets[s];
  const float* L = cell + 9 * s;
  int mx, my, mz;
  image_range(L, rc, mx, my, mz);
  const int ny = 2 * my + 1, nz = 2 * mz + 1;
  const int nimg = (2 * mx + 1) * ny * nz;
  const float xi = pos[3 * i], yi = pos[3 * i + 1], zi = pos[3 * i + 2];
  const float rc2 = __fmul_rn(rc, rc);
  const int b0 = bin_off[s];
  int cnt = 0;
  for (int im = 0; im < nimg; ++im) {
    const int ix = im / (ny * nz) - mx, iy = (im / nz) % ny - my, iz = im % nz - mz;
    float sx, sy, sz;
    image_shift(L, ix, iy, iz, sx, sy, sz);
    // atoms j near X_i - s(n): bins of the widened ball
    const double c[3] = {(double)xi - (double)sx, (double)yi - (double)sy, (double)zi - (double)sz};
    int lo[3], hi[3];
    bool empty = false;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      const double r = (double)rc + g.margin[k];
      empty |= c[k] + r < g.lo[k] || c[k] - r > g.hi[k];
      if (g.inv_w[k] == 0.0) {
        lo[k] = hi[k] = 0;
      } else {
        const double f0 = floor((c[k] - r - g.lo[k]) * g.inv_w[k]), f1 = floor((c[k] + r - g.lo[k]) * g.inv_w[k]);
        lo[k] = f0 < 0.0 ? 0 : f0 > g.nb[k] - 1 ? g.nb[k] - 1 : (int)f0;
        hi[k] = f1 < 0.0 ? 0 : f1 > g.nb[k] - 1 ? g.nb[k] - 1 : (int)f1;
      }
    }
    if (empty) continue;
    const bool zero_image = ix == 0 && iy == 0 && iz == 0;
    for (int bx = lo[0]; bx <= hi[0]; ++bx)
      for (int by = lo[1]; by <= hi[1]; ++by)
        for (int bz = lo[2]; bz <= hi[2]; ++bz) {
          const int b = b0 + (bx * g.nb[1] + by) * g.nb[2] + bz;
          const int r0 = bstart[b], r1 = bstart[b + 1];
          for (int t0 = r0; t0 < r1; t0 += 64) {
            const int t = t0 + lane;
            int j = 0;
            bool keep = false;
            if (t < r1) {
              j = batoms[t];
              keep = pair_kept(pos, i, j, xi, yi, zi, sx, sy, sz, zero_image, rc2);
            }
            const unsigned long long m = __ballot(keep);
            if (WRITE && keep) {
              const int p = cnt + __popcll(m & ((1ull << lane) - 1ull));
              if (p < kCellCap) keys[p] = (unsigned long long)(j - a) * (unsigned long long)nimg + (unsigned)im;
            }
            cnt += __popcll(m);
          }
        }
  }
  if (!WRITE) {
    if (lane == 0) count[i] = cnt;
    return;
  }
  cell_wave_sync();
  // rank of every key among the centre's keys (all distinct) = its place in the canonical order
  const int base = rowptr[i];
  for (int q = lane; q < cnt; q += 64) {
    const unsigned long long k = keys[q];
    int r = 0;
    for (int t = 0; t < cnt; ++t) r += keys[t] < k;
    const int p = base + r;
    const int j = a + (int)(k / (unsigned long long)nimg);
    const int im = (int)(k % (unsigned long long)nimg);
    ei[p] = i;
    ej[p] = j;
    shift[3 * p] = (int8_t)(im / (ny * nz) - mx);
    shift[3 * p + 1] = (int8_t)((im / nz) % ny - my);
    shift[3 * p + 2] = (int8_t)(im % nz - mz);
  }
}

// Exclusive scan of n int32 values into out[0..n]; out[n] is the total and
// totals that do not fit int32 raise flag bit 4.  Three passes over tiles of
// kScanTile values: tile sums, an exclusive scan of the tile sums (one
// workgroup), and the scan of every tile from its offset.  Sums are int64.
constexpr int kScanThreads = 256, kScanPer = 16, kScanTile = kScanThreads * kScanPer;

__device__ __forceinline__ long long block_exclusive_scan(long long v, long long* part, long long& total) {
  const int t = threadIdx.x;
  part[t] = v;
  __syncthreads();
  for (int o = 1; o < kScanThreads; o <<= 1) {
    const long long w = t >= o ? part[t - o] : 0;
    __syncthreads();
    part[t] += w;
    __syncthreads();
  }
  total = part[kScanThreads - 1];
  const long long r = part[t] - v;
  __syncthreads();
  return r;
}

__global__ void scan_tile_sums_kernel(const int* __restrict__ in, int n, long long* __restrict__ sums) {
  __shared__ long long part[kScanThreads];
  const long long lo = (long long)blockIdx.x * kScanTile + (long long)threadIdx.x * kScanPer;
  long long s = 0;
#pragma unroll
  for (int k = 0; k < kScanPer; ++k)
    if (lo + k < n) s += in[lo + k];
  long long total;
  block_exclusive_scan(s, part, total);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

__global__ void scan_sums_kernel(long long* __restrict__ sums, int ntiles, int n, int* __restrict__ out,
                                 int* __restrict__ flag) {
  __shared__ long long part[kScanThreads];
  const int per = (ntiles + kScanThreads - 1) / kScanThreads;
  const int lo = min(ntiles, (int)threadIdx.x * per), hi = min(ntiles, lo + per);
  long long s = 0;
  for (int k = lo; k < hi; ++k) s += sums[k];
  long long total;
  long long run = block_exclusive_scan(s, part, total);
  for (int k = lo; k < hi; ++k) {
    const long long v = sums[k];
    sums[k] = run;
    run += v;
  }
  if (threadIdx.x == 0) {
    out[n] = (int)total;
    if (total > 0x7fffffffLL && flag) atomicOr(flag, 16);
  }
}

__global__ void scan_tile_kernel(const int* __restrict__ in, int n, const long long* __restrict__ offs,
                                 int* __restrict__ out) {
  __shared__ long long part[kScanThreads];
  const long long lo = (long long)blockIdx.x * kScanTile + (long long)threadIdx.x * kScanPer;
  int v[kScanPer];
  long long s = 0;
#pragma unroll
  for (int k = 0; k < kScanPer; ++k) {
    v[k] = lo + k < n ? in[lo + k] : 0;
    s += v[k];
  }
  long long total;
  long long run = offs[blockIdx.x] + block_exclusive_scan(s, part, total);
#pragma unroll
  for (int k = 0; k < kScanPer; ++k) {
    if (lo + k < n) out[lo + k] = (int)run;
    run += v[k];
  }
}

// rev[e] = the edge (j, i, -n), found by binary search in the sorted segment of j.
__global__ void reverse_kernel(const int* __restrict__ ei, const int* __restrict__ ej,
                               const int8_t* __restrict__ shift, const int* __restrict__ rowptr, int Ne,
                               int* __restrict__ rev, int* __restrict__ flag) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= Ne) return;
  const int i = ei[e], j = ej[e];
  const int kx = -shift[3 * e], ky = -shift[3 * e + 1], kz = -shift[3 * e + 2];
  // key of an edge within the segment of j: (ej, sx, sy, sz) lexicographic
  auto less = [&](int f) {
    int fj = ej[f];
    if (fj != i) return fj < i;
    int fx = shift[3 * f], fy = shift[3 * f + 1], fz = shift[3 * f + 2];
    if (fx != kx) return fx < kx;
    if (fy != ky) return fy < ky;
    return fz < kz;
  };
  int lo = rowptr[j], hi = rowptr[j + 1];
  while (lo < hi) {
    int mid = (lo + hi) >> 1;
    if (less(mid)) lo = mid + 1; else hi = mid;
  }
  bool ok = lo < rowptr[j + 1] && ej[lo] == i && shift[3 * lo] == kx && shift[3 * lo + 1] == ky &&
            shift[3 * lo + 2] == kz;
  rev[e] = ok ? lo : e;
  if (!ok) atomicOr(flag, 8);
}

// Edge geometry in float64 from the fp32 inputs, then stored as fp32:
// d = X_j + n.L - X_i, r = |d|, u = d / r, and the Bessel basis with the p = 6
// polynomial envelope and its radial derivative,
//   B_n(r)  = sqrt(2/rc) sin(n pi r / rc) / r * u(r / rc),
//   u(x)    = 1 - 28 x^6 + 48 x^7 - 21 x^8   (x < 1).
// Envelope u(r / rc) and its radial derivative (zero beyond the cutoff).
__device__ __forceinline__ void envelope_at(double r, double rcd, double& u, double& du) {
  const double x = r / rcd;
  u = 0.0;
  du = 0.0;
  if (x < 1.0) {
    const double x2 = x * x, x5 = x2 * x2 * x, x6 = x5 * x;
    u = 1.0 - 28.0 * x6 + 48.0 * x6 * x - 21.0 * x6 * x2;
    du = (-168.0 * x5 + 336.0 * x6 - 168.0 * x6 * x) / rcd;
  }
}

// B_n(r) and dB_n/dr, n = 1..nb, for cutoff rc, into B[0..nb), dB[0..nb).
__device__ __forceinline__ void bessel_at(double r, double rcd, int nb, float* __restrict__ B,
                                          float* __restrict__ dB) {
  double u, du;
  envelope_at(r, rcd, u, du);
  const double c = sqrt(2.0 / rcd);
  const double th = M_PI / rcd;
  // sin(n x), cos(n x) for x = th r by the angle-addition identities from one sincos
  // (float64: the recurrence's rounding stays far below the float32 outputs')
  double s1, c1;
  sincos(th * r, &s1, &c1);
  double sn = s1, cs = c1;
  const double ir = 1.0 / r;
  // nb is a multiple of 4 and the rows 16-byte aligned: four values per store
  for (int n0 = 1; n0 <= nb; n0 += 4) {
    float b[4], db[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const double k = (n0 + q) * th;
      const double s = sn * ir;
      const double ds = (k * cs - s) * ir;
      b[q] = (float)(c * s * u);
      db[q] = (float)(c * (ds * u + s * du));
      const double sn1 = sn * c1 + cs * s1;
      cs = cs * c1 - sn * s1;
      sn = sn1;
    }
    *reinterpret_cast<float4*>(B + n0 - 1) = make_float4(b[0], b[1], b[2], b[3]);
    *reinterpret_cast<float4*>(dB + n0 - 1) = make_float4(db[0], db[1], db[2], db[3]);
  }
}

// d2B_n/dr2, n = 1..nb, for cutoff rc (the loss gradient in positions needs the
// second radial derivative of the basis):
//   B = c s u,  s = sin(k r) / r,  s' = (k cos(k r) - s) / r,  s'' = -k^2 s - 2 s' / r,
//   B'' = c (s'' u + 2 s' u' + s u''),  u'' = (-840 x^4 + 2016 x^5 - 1176 x^6) / rc^2.
__device__ __forceinline__ void bessel_d2_at(double r, double rcd, int nb, float* __restrict__ d2B) {
  double u, du;
  envelope_at(r, rcd, u, du);
  const double x = r / rcd;
  double d2u = 0.0;
  if (x < 1.0) {
    const double x2 = x * x, x4 = x2 * x2;
    d2u = (-840.0 * x4 + 2016.0 * x4 * x - 1176.0 * x4 * x2) / (rcd * rcd);
  }
  const double c = sqrt(2.0 / rcd);
  const double th = M_PI / rcd;
  double s1, c1;
  sincos(th * r, &s1, &c1);
  double sn = s1, cs = c1;
  const double ir = 1.0 / r;
  for (int n0 = 1; n0 <= nb; n0 += 4) {
    float b[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const double k = (n0 + q) * th;
      const double s = sn * ir;
      const double ds = (k * cs - s) * ir;
      const double d2s = -k * k * s - 2.0 * ds * ir;
      b[q] = (float)(c * (d2s * u + 2.0 * ds * du + s * d2u));
      const double sn1 = sn * c1 + cs * s1;
      cs = cs * c1 - sn * s1;
      sn = sn1;
    }
    *reinterpret_cast<float4*>(d2B + n0 - 1) = make_float4(b[0], b[1], b[2], b[3]);
  }
}

// With rc3 > 0 also the three-body basis B3, dB3 (cutoff rc3) and the
// envelope u(r / rc3) with its derivative, per edge; with d2B also B''.
__global__ void geometry_kernel(const float* __restrict__ pos, const float* __restrict__ cell,
                                const int* __restrict__ sid, const int* __restrict__ ei,
                                const int* __restrict__ ej, const int8_t* __restrict__ shift, int Ne,
                                float rc, int nb, float4* __restrict__ geo, float* __restrict__ B,
                                float* __restrict__ dB, float rc3, float* __restrict__ B3, float* __restrict__ dB3,
                                float* __restrict__ u3, float* __restrict__ du3, float* __restrict__ d2B) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= Ne) return;
  const int i = ei[e], j = ej[e];
  const float* L = cell + 9 * sid[i];
  const double nx = shift[3 * e], ny = shift[3 * e + 1], nz = shift[3 * e + 2];
  double d[3];
#pragma unroll
  for (int k = 0; k < 3; ++k)
    d[k] = ((double)pos[3 * j + k] - (double)pos[3 * i + k]) +
           (nx * (double)L[k] + ny * (double)L[3 + k] + nz * (double)L[6 + k]);
  const double r = sqrt(d[0] * d[0] + d[1] * d[1] + d[2] * d[2]);
  geo[e] = make_float4((float)(d[0] / r), (float)(d[1] / r), (float)(d[2] / r), (float)r);
  bessel_at(r, (double)rc, nb, B + (long long)e * nb, dB + (long long)e * nb);
  if (d2B) bessel_d2_at(r, (double)rc, nb, d2B + (long long)e * nb);
  if (rc3 > 0.f) {
    bessel_at(r, (double)rc3, nb, B3 + (long long)e * nb, dB3 + (long long)e * nb);
    double u, du;
    envelope_at(r, (double)rc3, u, du);
    u3[e] = (float)u;
    du3[e] = (float)du;
  }
}

void launch_validate_struct(hipStream_t st, const int* offsets, int S, int N, const float* cell, float rc,
                            int* flag) {
  hipLaunchKernelGGL(validate_struct_kernel, dim3(cdiv(S + 1, 256)), dim3(256), 0, st, offsets, S, N, cell,
                     rc, flag);
}

void launch_atom_struct(hipStream_t st, const int* offsets, int S, int N, int* sid) {
  hipLaunchKernelGGL(atom_struct_kernel, dim3(S), dim3(256), 0, st, offsets, S, N, sid);
}

// scratch: cdiv(n, kScanTile) int64 values (scan_scratch_bytes)
size_t scan_scratch_bytes(long long n) { return sizeof(long long) * (size_t)((n + kScanTile - 1) / kScanTile + 1); }

void launch_exclusive_scan(hipStream_t st, const int* in, int n, int* out, int* flag, long long* scratch) {
  const int ntiles = (int)cdiv(n, kScanTile);
  if (ntiles > 0) {
    hipLaunchKernelGGL(scan_tile_sums_kernel, dim3(ntiles), dim3(kScanThreads), 0, st, in, n, scratch);
  }
  hipLaunchKernelGGL(scan_sums_kernel, dim3(1), dim3(kScanThreads), 0, st, scratch, ntiles, n, out, flag);
  if (ntiles > 0) {
    hipLaunchKernelGGL(scan_tile_kernel, dim3(ntiles), dim3(kScanThreads), 0, st, in, n, (const long long*)scratch,
                       out);
  }
}

void launch_geometry(hipStream_t st, const float* pos, const float* cell, const int* sid, const int* ei,
                     const int* ej, const int8_t* shift, int Ne, float rc, int nb, float4* geo, float* B,
                     float* dB, float rc3, float* B3, float* dB3, float* u3, float* du3, float* d2B) {
  if (Ne <= 0) return;
  hipLaunchKernelGGL(geometry_kernel, dim3(cdiv(Ne, 256)), dim3(256), 0, st, pos, cell, sid, ei, ej, shift, Ne,
                     rc, nb, geo, B, dB, rc3, B3, dB3, u3, du3, d2B);
}

}  // namespace janus

using namespace janus;

extern "C" int janus_set_edge_builder(janus_ctx* ctx, int32_t mode) {
  if (!ctx || mode < 0 || mode > 2) return JANUS_EINVAL;
  ctx->edge_builder = mode;
  return JANUS_OK;
}

extern "C" int janus_build_edges(janus_ctx* ctx, const float* pos, const float* cell, const int32_t* offsets,
                                 int32_t n_atoms, int32_t n_struct, int64_t capacity, int32_t* ei, int32_t* ej,
                                 int8_t* shift, int32_t* rowptr, int32_t* rev, int64_t* n_edges, void* stream) {
  if (!ctx || !pos || !cell || !offsets || !rowptr || !n_edges || n_atoms < 1 || n_struct < 1 || capacity < 0)
    return JANUS_EINVAL;
  if (capacity > 0 && (!ei || !ej || !shift || !rev)) return JANUS_EINVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int N = n_atoms, S = n_struct;
  const long long scan_n = N > S ? N : S;
  auto carve = [&](Carver& c, int*& flag, int*& sid, int*& count, int*& rp, long long*& scan, CellGrid*& grid,
                   int*& nbins, int*& bin_off, int*& abin, int*& bcount, int*& bstart, int*& bfill, int*& batoms) {
    flag = c.take<int>(1);
    sid = c.take<int>(N);
    count = c.take<int>(N);
    rp = c.take<int>(N + 1);
    scan = c.take<long long>(scan_scratch_bytes(scan_n) / sizeof(long long));
    grid = c.take<CellGrid>(S);
    nbins = c.take<int>(S);
    bin_off = c.take<int>(S + 1);
    abin = c.take<int>(N);
    bcount = c.take<int>(N);
    bstart = c.take<int>(N + 1);
    bfill = c.take<int>(N);
    batoms = c.take<int>(N);
  };
  int *flag, *sid, *count, *rp, *nbins, *bin_off, *abin, *bcount, *bstart, *bfill, *batoms;
  long long* scan;
  CellGrid* grid;
  Carver cv(nullptr);
  carve(cv, flag, sid, count, rp, scan, grid, nbins, bin_off, abin, bcount, bstart, bfill, batoms);
  int rc = ensure(ctx->nl, cv.size());
  if (rc) return rc;
  Carver c2(ctx->nl.ptr);
  carve(c2, flag, sid, count, rp, scan, grid, nbins, bin_off, abin, bcount, bstart, bfill, batoms);
  int* hw = ctx->host_word;

  JANUS_HIP_TRY(hipMemsetAsync(flag, 0, sizeof(int), st));
  launch_validate_struct(st, offsets, S, N, cell, ctx->cfg.r_cut, flag);
  launch_atom_struct(st, offsets, S, N, sid);
  JANUS_HIP_TRY(hipGetLastError());
  JANUS_HIP_TRY(hipMemcpyAsync(hw, flag, sizeof(int), hipMemcpyDeviceToHost, st));
  JANUS_HIP_TRY(hipStreamSynchronize(st));
  if (hw[0] & 1) return JANUS_EINVAL;
  if (hw[0] & 2) return JANUS_EUNSUPPORTED;

  const float r_cut = ctx->cfg.r_cut;
  const dim3 gw(cdiv((long long)N * 64, 256)), b256(256);
  {
    ProfScope ps(ctx, st, PROF_GRAPH, 0.0, 16.0 * N);
    // cell lists of the structures that use them (none in mode 2)
    hipLaunchKernelGGL(cell_grid_kernel, dim3(S), b256, 0, st, pos, cell, offsets, S, r_cut, ctx->edge_builder, grid,
                       nbins);
    if (ctx->edge_builder != 2) {
      launch_exclusive_scan(st, nbins, S, bin_off, flag, scan);
      JANUS_HIP_TRY(hipMemsetAsync(bcount, 0, sizeof(int) * N, st));
      JANUS_HIP_TRY(hipMemsetAsync(bfill, 0, sizeof(int) * N, st));
      hipLaunchKernelGGL(cell_bin_kernel, dim3(cdiv(N, 256)), b256, 0, st, pos, sid, grid, bin_off, N, abin, bcount);
      launch_exclusive_scan(st, bcount, N, bstart, flag, scan);
      hipLaunchKernelGGL(cell_fill_kernel, dim3(cdiv(N, 256)), b256, 0, st, sid, grid, abin, bstart, N, bfill,
                         batoms);
      hipLaunchKernelGGL((nl_cell_kernel<false>), gw, b256, 0, st, pos, cell, offsets, sid, r_cut, N, grid, bin_off,
                         bstart, batoms, count, nullptr, nullptr, nullptr, nullptr);
    }
    hipLaunchKernelGGL((nl_kernel<false>), gw, b256, 0, st, pos, cell, offsets, sid, r_cut, N, count, nullptr,
                       nullptr, nullptr, nullptr, grid);
    launch_exclusive_scan(st, count, N, rp, flag, scan);
  }
  JANUS_HIP_TRY(hipGetLastError());
  JANUS_HIP_TRY(hipMemcpyAsync(hw, rp + N, sizeof(int), hipMemcpyDeviceToHost, st));
  JANUS_HIP_TRY(hipMemcpyAsync(hw + 1, flag, sizeof(int), hipMemcpyDeviceToHost, st));
  JANUS_HIP_TRY(hipStreamSynchronize(st));
  if (hw[1] & 16) return JANUS_EUNSUPPORTED;   // more than 2^31 - 1 edges
  const long long ne = hw[0];
  *n_edges = ne;
  if (ne > capacity) return JANUS_ECAPACITY;
  JANUS_HIP_TRY(hipMemcpyAsync(rowptr, rp, sizeof(int) * (N + 1), hipMemcpyDeviceToDevice, st));
  if (ne > 0) {
    ProfScope ps(ctx, st, PROF_GRAPH, 0.0, 16.0 * N + 23.0 * ne);
    if (ctx->edge_builder != 2)
      hipLaunchKernelGGL((nl_cell_kernel<true>), gw, b256, 0, st, pos, cell, offsets, sid, r_cut, N, grid, bin_off,
                         bstart, batoms, count, rp, ei, ej, shift);
    hipLaunchKernelGGL((nl_kernel<true>), gw, b256, 0, st, pos, cell, offsets, sid, r_cut, N, count, rp, ei, ej,
                       shift, grid);
    hipLaunchKernelGGL(reverse_kernel, dim3(cdiv(ne, 256)), dim3(256), 0, st, ei, ej, shift, rp, (int)ne, rev,
                       flag);
  }
  JANUS_HIP_TRY(hipGetLastError());
  return JANUS_OK;
}
