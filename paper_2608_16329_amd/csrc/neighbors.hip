// Cell-list neighbour builder for gfx950 (the binning step the paper takes
// from LAMMPS, Section 4.1; neighbour sets of Section 3.1).
//
// Atoms are binned into cells of edge >= cutoff + skin and counting-sorted by
// key = species * ncell + cell, so every (species, cell) bucket is a
// contiguous run of "sorted slots".  Each row is then found by scanning the
// 27 surrounding cells (deduplicated when a dimension has fewer than 3
// cells), species by species, which groups a row's entries by neighbour
// species.  The distance test is the exact one of the library's contract:
// wrapped coordinates, one minimum-image fold, (dx*dx + dy*dy) + dz*dz with
// round-to-nearest products and sums (no contraction), strict comparison.
#include "kernel_math.h"
#include "mlip_internal.h"

namespace mlip {
namespace {

constexpr int kScanThreads = 256;
constexpr int kScanItems = 8;
constexpr int kScanSeg = kScanThreads * kScanItems;

__device__ inline double wrap1(double x, double L) {
  double w = fmod(x, L);
  if (w < 0.0) w = w + L;
  if (w >= L) w = w - L;
  return w;
}

__device__ inline int cell_of(double w, double scale, int nc) {
  int c = int(w * scale);
  return c < nc ? c : nc - 1;
}

// Distinct periodic neighbours of cell c in a dimension of nc cells, in the
// order the coded entries refer to (nbr_cells); returns how many.
__device__ inline int adjacent(int c, int nc, int out[3]) {
  nbr_cells(c, nc, out);
  return nc >= 3 ? 3 : nc;
}

// Largest value over the wavefront (every lane active), applied by its first
// lane with one atomic.
__device__ inline void wave_atomic_max(int32_t* dst, int v) {
  for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, 64));
  if ((threadIdx.x & 63) == 0) atomicMax(dst, v);
}

__device__ inline double fold_half(double d, double L, double h) {
  if (d > h) return d - L;
  if (d < -h) return d + L;
  return d;
}

__device__ inline double sqdist(double dx, double dy, double dz) {
  return __dadd_rn(__dadd_rn(__dmul_rn(dx, dx), __dmul_rn(dy, dy)), __dmul_rn(dz, dz));
}

__global__ void k_bin(const double* __restrict__ pos, const int32_t* __restrict__ types, int64_t n,
                      NbrGrid g, int32_t* __restrict__ key, int32_t* __restrict__ cell_count,
                      int32_t* __restrict__ flags) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= n) return;
  double x = pos[3 * i], y = pos[3 * i + 1], z = pos[3 * i + 2];
  int t = types[i];
  const bool ok = t >= 0 && t < g.C && isfinite(x) && isfinite(y) && isfinite(z);
  if (!ok) {
    atomicOr(&flags[0], 1);
    t = 0;
    x = y = z = 0.0;
  }
  const int cx = cell_of(wrap1(x, g.box[0]), g.cell_scale[0], g.nc[0]);
  const int cy = cell_of(wrap1(y, g.box[1]), g.cell_scale[1], g.nc[1]);
  const int cz = cell_of(wrap1(z, g.box[2]), g.cell_scale[2], g.nc[2]);
  const int k = t * g.ncell + (cz * g.nc[1] + cy) * g.nc[0] + cx;
  key[i] = k;
  atomicAdd(&cell_count[k], 1);
}

// Counting-sort scatter; flags[2] receives the largest bucket (which decides
// whether entries fit the 16-bit code).
__global__ void k_scatter(const int32_t* __restrict__ key, int64_t n, const int32_t* __restrict__ start,
                          int32_t* __restrict__ fill, int32_t* __restrict__ perm, int32_t* __restrict__ flags) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if ((i & ~int64_t(63)) >= n) return;  // the whole wavefront is past the end
  int place = 0;
  if (i < n) {
    const int k = key[i];
    place = atomicAdd(&fill[k], 1);
    perm[start[k] + place] = int32_t(i);
  }
  wave_atomic_max(&flags[2], place + 1);
}

// Make the order inside each (species, cell) bucket deterministic.
__global__ void k_sort_segments(const int32_t* __restrict__ start, int64_t nkeys, int32_t* __restrict__ perm) {
  const int64_t k = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (k >= nkeys) return;
  const int b = start[k], e = start[k + 1];
  for (int i = b + 1; i < e; ++i) {
    const int v = perm[i];
    int j = i - 1;
    while (j >= b && perm[j] > v) {
      perm[j + 1] = perm[j];
      --j;
    }
    perm[j + 1] = v;
  }
}

__global__ void k_gather_sorted(const double* __restrict__ pos, const int32_t* __restrict__ perm, int64_t n,
                                NbrGrid g, double* __restrict__ spos) {
  const int64_t a = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (a >= n) return;
  const int64_t i = perm[a];
  spos[3 * a] = wrap1(pos[3 * i], g.box[0]);
  spos[3 * a + 1] = wrap1(pos[3 * i + 1], g.box[1]);
  spos[3 * a + 2] = wrap1(pos[3 * i + 2], g.box[2]);
}

// Rows by a 27-cell scan: the count pass (kFill false) records row lengths,
// the fill pass writes caller indices or, with kCode, 16-bit codes (ListView):
// a candidate's code names the scanned cell it sits in (tracked along each
// run of consecutive cells), its species and its place in that bucket.
template <bool kFill, bool kCode>
__global__ void k_rows(const double* __restrict__ spos, const int32_t* __restrict__ perm, int64_t n, NbrGrid g,
                       const int32_t* __restrict__ start, int32_t* __restrict__ rowcnt,
                       const int64_t* __restrict__ offsets, void* __restrict__ idx,
                       int32_t* __restrict__ flags, int tbits, int sbits) {
  const int64_t a0 = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if ((a0 & ~int64_t(63)) >= n) return;  // the whole wavefront is past the end
  if (kFill && a0 >= n) return;
  // count pass: lanes past the end repeat the last atom so that every lane
  // joins the wavefront's maximum
  const int64_t a = a0 < n ? a0 : n - 1;
  const double wx = spos[3 * a], wy = spos[3 * a + 1], wz = spos[3 * a + 2];
  int xs[3], ys[3], zs[3];
  const int nx = adjacent(cell_of(wx, g.cell_scale[0], g.nc[0]), g.nc[0], xs);
  const int ny = adjacent(cell_of(wy, g.cell_scale[1], g.nc[1]), g.nc[1], ys);
  const int nz = adjacent(cell_of(wz, g.cell_scale[2], g.nc[2]), g.nc[2], zs);
  int cnt = 0;
  const int64_t base = kFill ? offsets[a] : 0;
  for (int s = 0; s < g.C; ++s) {
    for (int iz = 0; iz < nz; ++iz)
      for (int iy = 0; iy < ny; ++iy) {
        // x-neighbour cells with consecutive indices are consecutive keys, so
        // their atoms form one run of the sorted order: visit runs, not cells
        // (same entries in the same order)
        int ix = 0;
        while (ix < nx) {
          const int ix0 = ix;
          const int x0 = xs[ix];
          int x1 = x0;
          while (ix + 1 < nx && xs[ix + 1] == x1 + 1) {
            ++ix;
            ++x1;
          }
          ++ix;
          const int key = s * g.ncell + (zs[iz] * g.nc[1] + ys[iy]) * g.nc[0] + x0;
          const int e = start[key + (x1 - x0) + 1];
          int cur = 0;                   // cell x0 + cur of the run holds slot b
          int cell_end = start[key + 1];
          for (int b = start[key]; b < e; ++b) {
            if (kCode)
              while (b >= cell_end) {
                ++cur;
                cell_end = start[key + cur + 1];
              }
            if (b == a) continue;
            const double dx = fold_half(spos[3 * int64_t(b)] - wx, g.box[0], g.half[0]);
            const double dy = fold_half(spos[3 * int64_t(b) + 1] - wy, g.box[1], g.half[1]);
            const double dz = fold_half(spos[3 * int64_t(b) + 2] - wz, g.box[2], g.half[2]);
            if (sqdist(dx, dy, dz) < g.rl2) {
              if (kFill) {
                if constexpr (kCode) {
                  const unsigned o = unsigned((iz * 3 + iy) * 3 + ix0 + cur);
                  const unsigned t = unsigned(b - start[key + cur]);
                  static_cast<uint16_t*>(idx)[base + cnt] =
                      uint16_t((o << (sbits + tbits)) | (unsigned(s) << tbits) | t);
                } else {
                  static_cast<int32_t*>(idx)[base + cnt] = perm[b];
                }
              }
              ++cnt;
            }
          }
        }
      }
  }
  if (!kFill) {
    if (a0 < n) rowcnt[a] = cnt;
    wave_atomic_max(&flags[1], cnt);
  }
}

// ---- exclusive scan: out[0..n] with out[n] = total -------------------------
template <typename Tin>
__global__ void k_block_sums(const Tin* __restrict__ in, int64_t n, int64_t* __restrict__ bsum) {
  __shared__ int64_t red[kScanThreads / 64];
  const int64_t base = int64_t(blockIdx.x) * kScanSeg;
  int64_t s = 0;
  for (int it = 0; it < kScanItems; ++it) {
    const int64_t i = base + int64_t(it) * kScanThreads + threadIdx.x;
    if (i < n) s += int64_t(in[i]);
  }
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t t = 0;
    for (int w = 0; w < kScanThreads / 64; ++w) t += red[w];
    bsum[blockIdx.x] = t;
  }
}

__device__ inline int64_t wave_inclusive(int64_t v) {
  const int lane = threadIdx.x & 63;
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t t = __shfl_up(v, o, 64);
    if (lane >= o) v += t;
  }
  return v;
}

// Exclusive scan of the block sums in place (single work-group, any length).
__global__ void k_scan_sums(int64_t* __restrict__ bsum, int64_t nb) {
  __shared__ int64_t wtot[kScanThreads / 64];
  __shared__ int64_t carry;
  if (threadIdx.x == 0) carry = 0;
  __syncthreads();
  for (int64_t b0 = 0; b0 < nb; b0 += kScanThreads) {
    const int64_t i = b0 + threadIdx.x;
    const int64_t v = i < nb ? bsum[i] : 0;
    const int64_t inc = wave_inclusive(v);
    if ((threadIdx.x & 63) == 63) wtot[threadIdx.x >> 6] = inc;
    __syncthreads();
    int64_t off = carry;
    for (int w = 0; w < int(threadIdx.x >> 6); ++w) off += wtot[w];
    if (i < nb) bsum[i] = off + inc - v;
    __syncthreads();
    if (threadIdx.x == kScanThreads - 1) carry = off + inc;
    __syncthreads();
  }
}

template <typename Tin, typename Tout>
__global__ void k_scan_apply(const Tin* __restrict__ in, int64_t n, const int64_t* __restrict__ bsum,
                             Tout* __restrict__ out) {
  __shared__ int64_t wtot[kScanThreads / 64];
  const int64_t base = int64_t(blockIdx.x) * kScanSeg + int64_t(threadIdx.x) * kScanItems;
  int64_t v[kScanItems];
  int64_t tsum = 0;
  for (int it = 0; it < kScanItems; ++it) {
    const int64_t i = base + it;
    v[it] = i < n ? int64_t(in[i]) : 0;
    tsum += v[it];
  }
  const int64_t inc = wave_inclusive(tsum);
  if ((threadIdx.x & 63) == 63) wtot[threadIdx.x >> 6] = inc;
  __syncthreads();
  int64_t run = bsum[blockIdx.x] + inc - tsum;
  for (int w = 0; w < int(threadIdx.x >> 6); ++w) run += wtot[w];
  for (int it = 0; it < kScanItems; ++it) {
    const int64_t i = base + it;
    if (i < n) out[i] = Tout(run);
    run += v[it];
    if (i == n - 1) out[n] = Tout(run);
  }
}

template <typename T>
__global__ void k_fill(T* __restrict__ p, int64_t n, T v) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

template <typename Tin, typename Tout>
hipError_t exclusive_scan(const Tin* in, int64_t n, Tout* out, int64_t* tmp, hipStream_t s) {
  if (n == 0) {
    k_fill<Tout><<<1, 1, 0, s>>>(out, 1, Tout(0));
    return hipGetLastError();
  }
  const int64_t nb = (n + kScanSeg - 1) / kScanSeg;
  k_block_sums<Tin><<<dim3(unsigned(nb)), dim3(kScanThreads), 0, s>>>(in, n, tmp);
  k_scan_sums<<<1, kScanThreads, 0, s>>>(tmp, nb);
  k_scan_apply<Tin, Tout><<<dim3(unsigned(nb)), dim3(kScanThreads), 0, s>>>(in, n, tmp, out);
  return hipGetLastError();
}

inline unsigned blocks_for(int64_t n, int t) { return unsigned((n + t - 1) / t); }

}  // namespace

size_t scan_tmp_elems(int64_t n) { return size_t((n + kScanSeg - 1) / kScanSeg) + 1; }

hipError_t launch_exclusive_scan_i32_to_i32(const int32_t* in, int64_t n, int32_t* out, int64_t* tmp,
                                            hipStream_t s) {
  return exclusive_scan<int32_t, int32_t>(in, n, out, tmp, s);
}

hipError_t launch_exclusive_scan_i32_to_i64(const int32_t* in, int64_t n, int64_t* out, int64_t* tmp,
                                            hipStream_t s) {
  return exclusive_scan<int32_t, int64_t>(in, n, out, tmp, s);
}

hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  k_fill<int32_t><<<blocks_for(n, 256), 256, 0, s>>>(p, n, v);
  return hipGetLastError();
}

hipError_t launch_fill_f64(double* p, int64_t n, double v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  k_fill<double><<<blocks_for(n, 256), 256, 0, s>>>(p, n, v);
  return hipGetLastError();
}

hipError_t launch_fill_u64(unsigned long long* p, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  k_fill<unsigned long long><<<blocks_for(n, 256), 256, 0, s>>>(p, n, 0ull);
  return hipGetLastError();
}

hipError_t launch_bin(const double* pos, const int32_t* types, int64_t n, const NbrGrid& g, int32_t* key,
                      int32_t* cell_count, int32_t* flags, hipStream_t s) {
  k_bin<<<blocks_for(n, 256), 256, 0, s>>>(pos, types, n, g, key, cell_count, flags);
  return hipGetLastError();
}

hipError_t launch_scatter(const int32_t* key, int64_t n, const int32_t* cell_start, int32_t* fill, int32_t* perm,
                          int32_t* flags, hipStream_t s) {
  k_scatter<<<blocks_for(n, 256), 256, 0, s>>>(key, n, cell_start, fill, perm, flags);
  return hipGetLastError();
}

hipError_t launch_sort_segments(const int32_t* cell_start, int64_t nkeys, int32_t* perm, hipStream_t s) {
  k_sort_segments<<<blocks_for(nkeys, 256), 256, 0, s>>>(cell_start, nkeys, perm);
  return hipGetLastError();
}

hipError_t launch_gather_sorted(const double* pos, const int32_t* perm, int64_t n, const NbrGrid& g,
                                double* spos, hipStream_t s) {
  k_gather_sorted<<<blocks_for(n, 256), 256, 0, s>>>(pos, perm, n, g, spos);
  return hipGetLastError();
}

hipError_t launch_rows(const double* spos, const int32_t* perm, int64_t n, const NbrGrid& g,
                       const int32_t* cell_start, int32_t* rowcnt, const int64_t* offsets, void* idx,
                       int32_t* flags, bool fill, int tbits, int sbits, hipStream_t s) {
  const unsigned nb = blocks_for(n, 128);
  if (!fill)
    k_rows<false, false><<<nb, 128, 0, s>>>(spos, perm, n, g, cell_start, rowcnt, offsets, idx, flags, 0, 0);
  else if (tbits > 0)
    k_rows<true, true><<<nb, 128, 0, s>>>(spos, perm, n, g, cell_start, rowcnt, offsets, idx, flags, tbits, sbits);
  else
    k_rows<true, false><<<nb, 128, 0, s>>>(spos, perm, n, g, cell_start, rowcnt, offsets, idx, flags, 0, 0);
  return hipGetLastError();
}

}  // namespace mlip
