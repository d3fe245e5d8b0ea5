// Device helpers shared by the kernel files: the periodic minimum-image fold
// and the Cartesian monomials of a unit vector with their gradients, over
// which the angular features are expanded (Eq. 3, Section 3.3).
#pragma once

#include <hip/hip_runtime.h>

#include "mlip_internal.h"

namespace mlip {

// Minimum-image fold of one coordinate difference (Eq. 1 in a periodic box).
__device__ __forceinline__ double fold(double d, double L, double invL) { return d - L * rint(d * invL); }

// The cells scanned around cell c in a dimension of nc cells, in scan order:
// c-1, c, c+1 (periodic) when nc >= 3, all cells otherwise.  Shared by the
// list builder and every reader of coded entries.
__host__ __device__ __forceinline__ void nbr_cells(int c, int nc, int out[3]) {
  if (nc >= 3) {
    out[0] = c == 0 ? nc - 1 : c - 1;
    out[1] = c;
    out[2] = c == nc - 1 ? 0 : c + 1;
  } else {
    out[0] = 0;
    out[1] = nc == 2 ? 1 : 0;
    out[2] = out[1];
  }
}

// The 3 x 3 candidate cells of a centre atom from its bucket key:
// cand[0..2] along x, [3..5] along y, [6..8] along z.
__host__ __device__ __forceinline__ void centre_cells(const ListView& L, int key, int cand[9]) {
  const int cell = key % L.ncell;
  const int cx = cell % L.nc[0], cy = (cell / L.nc[0]) % L.nc[1], cz = cell / (L.nc[0] * L.nc[1]);
  nbr_cells(cx, L.nc[0], cand);
  nbr_cells(cy, L.nc[1], cand + 3);
  nbr_cells(cz, L.nc[2], cand + 6);
}

// Sorted slot of a coded entry of a centre with candidate cells cand.
__host__ __device__ __forceinline__ int code_slot(const ListView& L, const int cand[9], unsigned code) {
  const int t = int(code & ((1u << L.tbits) - 1u));
  const int sp = int((code >> L.tbits) & ((1u << L.sbits) - 1u));
  const int o = int(code >> (L.tbits + L.sbits));
  const int ix = o % 3, iy = (o / 3) % 3, iz = o / 9;
  const int key = sp * L.ncell + (cand[6 + iz] * L.nc[1] + cand[3 + iy]) * L.nc[0] + cand[ix];
  return L.start[key] + t;
}

// Caller index of neighbour-list entry e of a centre (cand from centre_cells);
// the host readers of the list use it on host copies of the arrays.
__host__ __device__ __forceinline__ int list_entry(const ListView& L, const int cand[9], long long e) {
  if (L.idx32) return L.idx32[e];
  return L.perm[code_slot(L, cand, L.idx16[e])];
}

// Cartesian monomials of degree <= 3 in the order of the angular table
// (degree by degree, lexicographic with x first).
template <typename R>
__device__ __forceinline__ void monomials(R x, R y, R z, R m[kMonomials]) {
  m[0] = R(1);
  m[1] = x; m[2] = y; m[3] = z;
  m[4] = x * x; m[5] = x * y; m[6] = x * z; m[7] = y * y; m[8] = y * z; m[9] = z * z;
  m[10] = x * x * x; m[11] = x * x * y; m[12] = x * x * z; m[13] = x * y * y; m[14] = x * y * z;
  m[15] = x * z * z; m[16] = y * y * y; m[17] = y * y * z; m[18] = y * z * z; m[19] = z * z * z;
}

// Gradients of the monomials with respect to (x, y, z).
template <typename R>
__device__ __forceinline__ void monomial_grads(R x, R y, R z, R gx[kMonomials], R gy[kMonomials],
                                               R gz[kMonomials]) {
  const R xx = x * x, yy = y * y, zz = z * z;
  gx[0] = 0; gy[0] = 0; gz[0] = 0;
  gx[1] = 1; gy[1] = 0; gz[1] = 0;
  gx[2] = 0; gy[2] = 1; gz[2] = 0;
  gx[3] = 0; gy[3] = 0; gz[3] = 1;
  gx[4] = 2 * x; gy[4] = 0; gz[4] = 0;
  gx[5] = y; gy[5] = x; gz[5] = 0;
  gx[6] = z; gy[6] = 0; gz[6] = x;
  gx[7] = 0; gy[7] = 2 * y; gz[7] = 0;
  gx[8] = 0; gy[8] = z; gz[8] = y;
  gx[9] = 0; gy[9] = 0; gz[9] = 2 * z;
  gx[10] = 3 * xx; gy[10] = 0; gz[10] = 0;
  gx[11] = 2 * x * y; gy[11] = xx; gz[11] = 0;
  gx[12] = 2 * x * z; gy[12] = 0; gz[12] = xx;
  gx[13] = yy; gy[13] = 2 * x * y; gz[13] = 0;
  gx[14] = y * z; gy[14] = x * z; gz[14] = x * y;
  gx[15] = zz; gy[15] = 0; gz[15] = 2 * x * z;
  gx[16] = 0; gy[16] = 3 * yy; gz[16] = 0;
  gx[17] = 0; gy[17] = 2 * y * z; gz[17] = yy;
  gx[18] = 0; gy[18] = zz; gz[18] = 2 * y * z;
  gx[19] = 0; gy[19] = 0; gz[19] = 3 * zz;
}

}  // namespace mlip
