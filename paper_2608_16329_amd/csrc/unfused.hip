// The unfused configuration of the evaluation (Section 3.4, Table
// "Configurable fusion", row "before fusion"): one kernel per equation of
// Eqs. 1-10, every intermediate tensor in HBM (Section 3.1, "Major Sources of
// HBM Footprint": the per-pair g_rad, g_ang with their Jacobians, U_i and
// V_i, and the per-atom P_i, G_i and W_i).  It exists to measure what fusion
// buys on this GPU; results equal the fused kernel's up to rounding.
//
// This file holds eight of the ten kernels: setup (Eq. 1), angular features
// (Eq. 3), moment (Eq. 4), descriptor (Eq. 5), adjoint W (Eq. 7), U (Eq. 8),
// V (Eq. 9) and forces (Eq. 10).  The radial encoder (Eq. 2) and the head
// (Eq. 6) are dense contractions over 16-pair and 16-atom tiles and run as
// modes of the fused kernel's MFMA code.
//
// Per-entry arrays are indexed by the neighbour-list entry (rows of the
// sorted atoms, entries beyond the cutoff marked by r = -1 and skipped),
// per-atom arrays by sorted slot.  Per-atom kernels give one wavefront to
// one atom's row.  Only k = 32 and the irreducible basis with l_max <= 3
// (16 angular rows over 20 monomials) are built.
#include "kernel_math.h"
#include "mlip_internal.h"

namespace mlip {
namespace {

constexpr int K = 32;            // radial width
constexpr int D = kAngRows;      // angular rows (padded to 16)
constexpr int NM = kMonomials;   // monomials of degree <= 3
constexpr int kBlock = 256;      // threads per work-group: four wavefronts
constexpr int kAtomsPerBlock = kBlock / 64;

// Sorted slot of this wavefront's atom (one wavefront per atom), or -1.
__device__ __forceinline__ long long wave_atom(long long n) {
  const long long a = (long long)blockIdx.x * kAtomsPerBlock + (threadIdx.x >> 6);
  return a < n ? a : -1;
}

// Eq. 1: r_ij = r_j - r_i (minimum image), r = |r_ij|; r = -1 marks a listed
// entry at or beyond the cutoff (the same squared-distance test as the fused
// kernel's staging).
__global__ __launch_bounds__(kBlock) void k_setup(UnfusedArgs A) {
  const long long a = wave_atom(A.n);
  if (a < 0) return;
  const int lane = threadIdx.x & 63;
  const long long o = A.perm[a];
  const double xi = A.pos[3 * o], yi = A.pos[3 * o + 1], zi = A.pos[3 * o + 2];
  int cand[9];
  if (A.list.idx16) centre_cells(A.list, A.list.key[o], cand);
  const long long e1 = A.offsets[a + 1];
  for (long long e = A.offsets[a] + lane; e < e1; e += 64) {
    const long long j = list_entry(A.list, cand, e);
    const double dx = fold(A.pos[3 * j] - xi, A.box[0], A.inv_box[0]);
    const double dy = fold(A.pos[3 * j + 1] - yi, A.box[1], A.inv_box[1]);
    const double dz = fold(A.pos[3 * j + 2] - zi, A.box[2], A.inv_box[2]);
    const double d2 = dx * dx + dy * dy + dz * dz;
    double4 v;
    v.x = dx;
    v.y = dy;
    v.z = dz;
    v.w = d2 < A.rc2 ? sqrt(d2) : -1.0;
    reinterpret_cast<double4*>(A.geo)[e] = v;
  }
}

// Eq. 3 and its Jacobian: a = Q m(u) over the monomials of u = r_ij / r, and
// da/dr_ij = (I - u u^T) (grad_u a) / r; one thread per entry.
template <typename R>
__global__ __launch_bounds__(kBlock) void k_angular(UnfusedArgs A) {
  const long long e = (long long)blockIdx.x * kBlock + threadIdx.x;
  if (e >= A.n_entries) return;
  const double4 v = reinterpret_cast<const double4*>(A.geo)[e];
  if (v.w < 0.0) return;
  const R* __restrict__ qc = static_cast<const R*>(A.qc);
  const R r = R(v.w), ir = R(1) / r;
  const R ux = R(v.x) * ir, uy = R(v.y) * ir, uz = R(v.z) * ir;
  R mono[NM], gx[NM], gy[NM], gz[NM];
  monomials(ux, uy, uz, mono);
  monomial_grads(ux, uy, uz, gx, gy, gz);
  R* __restrict__ ga = static_cast<R*>(A.gang) + e * D;
  R* __restrict__ ja = static_cast<R*>(A.jang) + e * D * 3;
#pragma unroll
  for (int m = 0; m < D; ++m) {
    R s = 0, sx = 0, sy = 0, sz = 0;
#pragma unroll
    for (int t = 0; t < NM; ++t) {
      const R q = qc[m * NM + t];
      s += q * mono[t];
      sx += q * gx[t];
      sy += q * gy[t];
      sz += q * gz[t];
    }
    const R us = ux * sx + uy * sy + uz * sz;
    ga[m] = s;
    ja[3 * m] = (sx - us * ux) * ir;
    ja[3 * m + 1] = (sy - us * uy) * ir;
    ja[3 * m + 2] = (sz - us * uz) * ir;
  }
}

// Eq. 4: P_i = sum_j g_ang (x) g_rad over the atom's active entries; lane
// (m, c0) accumulates P[m][c0 .. c0+7].
template <typename R>
__global__ __launch_bounds__(kBlock) void k_moment(UnfusedArgs A) {
  const long long a = wave_atom(A.n);
  if (a < 0) return;
  const int lane = threadIdx.x & 63, m = lane >> 2, c0 = (lane & 3) * 8;
  const R* __restrict__ ga = static_cast<const R*>(A.gang);
  const R* __restrict__ gr = static_cast<const R*>(A.grad);
  R acc[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) acc[q] = 0;
  const long long e1 = A.offsets[a + 1];
  for (long long e = A.offsets[a]; e < e1; ++e) {
    if (A.geo[4 * e + 3] < 0.0) continue;
    const R am = ga[e * D + m];
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[q] += am * gr[e * K + c0 + q];
  }
  R* __restrict__ P = static_cast<R*>(A.P) + a * D * K;
#pragma unroll
  for (int q = 0; q < 8; ++q) P[m * K + c0 + q] = acc[q];
}

// Eq. 5: G[l][c] = P[0][c] for l = 0, sum over the order-l rows m of
// C_l[m] P[m][c]^2 otherwise; one thread per descriptor entry.
template <typename R>
__global__ __launch_bounds__(kBlock) void k_descriptor(UnfusedArgs A) {
  const int nin = (A.lmax + 1) * K;
  const long long u = (long long)blockIdx.x * kBlock + threadIdx.x;
  if (u >= A.n * nin) return;
  const long long a = u / nin;
  const int in = int(u % nin), l = in / K, c = in % K;
  const R* __restrict__ P = static_cast<const R*>(A.P) + a * D * K;
  const R* __restrict__ rw = static_cast<const R*>(A.qc) + D * NM;
  R v;
  if (l == 0) {
    v = P[c];
  } else {
    v = 0;
    for (int m = A.lrow[l]; m < A.lrow[l + 1]; ++m) v += rw[m] * P[m * K + c] * P[m * K + c];
  }
  static_cast<R*>(A.G)[u] = v;
}

// Eq. 7 through the descriptor: W[0][c] = dE/dG[0][c] and W[m][c] =
// 2 C_l[m] dE/dG[l][c] P[m][c] for a row m of order l >= 1; zero on the
// padding rows.  One thread per element of W.
template <typename R>
__global__ __launch_bounds__(kBlock) void k_adjoint(UnfusedArgs A) {
  const int nin = (A.lmax + 1) * K;
  const long long u = (long long)blockIdx.x * kBlock + threadIdx.x;
  if (u >= A.n * D * K) return;
  const long long a = u / (D * K);
  const int m = int(u % (D * K)) / K, c = int(u % K);
  const R* __restrict__ dG = static_cast<const R*>(A.G) + a * nin;
  const R* __restrict__ rw = static_cast<const R*>(A.qc) + D * NM;
  R w = 0;
  if (m == 0) {
    w = dG[c];
  } else if (m < A.lrow[A.lmax + 1]) {
    int l = 1;
    while (m >= A.lrow[l + 1]) ++l;
    w = R(2) * rw[m] * dG[l * K + c] * static_cast<const R*>(A.P)[u];
  }
  static_cast<R*>(A.W)[u] = w;
}

// Eq. 8: U_i = G_ang,i W_i, row j: u[c] = sum_m g_ang[m] W[m][c].  Lane
// (half, c) holds column c of W and takes every second entry.
template <typename R>
__global__ __launch_bounds__(kBlock) void k_u(UnfusedArgs A) {
  const long long a = wave_atom(A.n);
  if (a < 0) return;
  const int lane = threadIdx.x & 63, half = lane >> 5, c = lane & 31;
  const R* __restrict__ W = static_cast<const R*>(A.W) + a * D * K;
  R w[D];
#pragma unroll
  for (int m = 0; m < D; ++m) w[m] = W[m * K + c];
  const R* __restrict__ ga = static_cast<const R*>(A.gang);
  R* __restrict__ U = static_cast<R*>(A.U);
  const long long e1 = A.offsets[a + 1];
  for (long long e = A.offsets[a] + half; e < e1; e += 2) {
    if (A.geo[4 * e + 3] < 0.0) continue;
    R s = 0;
#pragma unroll
    for (int m = 0; m < D; ++m) s += ga[e * D + m] * w[m];
    U[e * K + c] = s;
  }
}

// Eq. 9: V_i = G_rad,i W_i^T, row j: v[m] = sum_c g_rad[c] W[m][c].  Lane
// (quarter, m) holds row m of W and takes every fourth entry.
template <typename R>
__global__ __launch_bounds__(kBlock) void k_v(UnfusedArgs A) {
  const long long a = wave_atom(A.n);
  if (a < 0) return;
  const int lane = threadIdx.x & 63, quarter = lane >> 4, m = lane & 15;
  const R* __restrict__ W = static_cast<const R*>(A.W) + a * D * K;
  R w[K];
#pragma unroll
  for (int c = 0; c < K; ++c) w[c] = W[m * K + c];
  const R* __restrict__ gr = static_cast<const R*>(A.grad);
  R* __restrict__ V = static_cast<R*>(A.V);
  const long long e1 = A.offsets[a + 1];
  for (long long e = A.offsets[a] + quarter; e < e1; e += 4) {
    if (A.geo[4 * e + 3] < 0.0) continue;
    R s = 0;
#pragma unroll
    for (int c = 0; c < K; ++c) s += gr[e * K + c] * w[c];
    V[e * D + m] = s;
  }
}

// Eq. 10: f_ij = J_rad^T u + J_ang^T v with J_rad = (dg_rad/dr) u_hat^T, so
// f = (g' . u) u_hat + sum_m v[m] dg_ang[m]/dr_ij; then F_i += f, F_j -= f,
// w_i -= r_ij (x) f (Section 3.1, scatter-sum), in float64.  Lanes take the
// atom's entries; F_i and w_i are summed across the wavefront.
template <typename R>
__global__ __launch_bounds__(kBlock) void k_force(UnfusedArgs A) {
  const long long a = wave_atom(A.n);
  if (a < 0) return;
  const int lane = threadIdx.x & 63;
  const R* __restrict__ gp = static_cast<const R*>(A.gprime);
  const R* __restrict__ U = static_cast<const R*>(A.U);
  const R* __restrict__ V = static_cast<const R*>(A.V);
  const R* __restrict__ ja = static_cast<const R*>(A.jang);
  double fi[3] = {0, 0, 0}, wi[9] = {0, 0, 0, 0, 0, 0, 0, 0, 0};
  int cand[9];
  if (A.list.idx16) centre_cells(A.list, A.list.key[A.perm[a]], cand);
  const long long e1 = A.offsets[a + 1];
  for (long long e = A.offsets[a] + lane; e < e1; e += 64) {
    const double4 v = reinterpret_cast<const double4*>(A.geo)[e];
    if (v.w < 0.0) continue;
    R s = 0;
#pragma unroll
    for (int c = 0; c < K; ++c) s += gp[e * K + c] * U[e * K + c];
    R tx = 0, ty = 0, tz = 0;
#pragma unroll
    for (int m = 0; m < D; ++m) {
      const R vm = V[e * D + m];
      tx += vm * ja[(e * D + m) * 3];
      ty += vm * ja[(e * D + m) * 3 + 1];
      tz += vm * ja[(e * D + m) * 3 + 2];
    }
    const R ir = R(1) / R(v.w);
    const double f[3] = {double(s * R(v.x) * ir + tx), double(s * R(v.y) * ir + ty), double(s * R(v.z) * ir + tz)};
    const long long j = list_entry(A.list, cand, e);
#pragma unroll
    for (int d = 0; d < 3; ++d) {
      atomicAdd(&A.forces[3 * j + d], -f[d]);
      fi[d] += f[d];
    }
    const double rv[3] = {v.x, v.y, v.z};
#pragma unroll
    for (int p = 0; p < 3; ++p)
#pragma unroll
      for (int q = 0; q < 3; ++q) wi[3 * p + q] -= rv[p] * f[q];
  }
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
#pragma unroll
    for (int d = 0; d < 3; ++d) fi[d] += __shfl_xor(fi[d], o, 64);
#pragma unroll
    for (int k = 0; k < 9; ++k) wi[k] += __shfl_xor(wi[k], o, 64);
  }
  if (lane == 0) {
    const long long o = A.perm[a];
#pragma unroll
    for (int d = 0; d < 3; ++d) atomicAdd(&A.forces[3 * o + d], fi[d]);
    if (A.virial)
#pragma unroll
      for (int k = 0; k < 9; ++k) A.virial[9 * o + k] = wi[k];
#pragma unroll
    for (int k = 0; k < 9; ++k) atomicAdd(&A.totals[1 + k], wi[k]);
  }
}

template <typename R>
hipError_t launch_stage(int stage, const UnfusedArgs& a, hipStream_t s) {
  const unsigned per_atom = unsigned((a.n + kAtomsPerBlock - 1) / kAtomsPerBlock);
  const unsigned per_entry = unsigned((a.n_entries + kBlock - 1) / kBlock);
  const long long nin = (a.lmax + 1) * K;
  const unsigned per_g = unsigned((a.n * nin + kBlock - 1) / kBlock);
  const unsigned per_w = unsigned((a.n * D * K + kBlock - 1) / kBlock);
  switch (stage) {
    case kUnfSetup: k_setup<<<per_atom, kBlock, 0, s>>>(a); break;
    case kUnfAngular: if (per_entry) k_angular<R><<<per_entry, kBlock, 0, s>>>(a); break;
    case kUnfMoment: k_moment<R><<<per_atom, kBlock, 0, s>>>(a); break;
    case kUnfDescriptor: k_descriptor<R><<<per_g, kBlock, 0, s>>>(a); break;
    case kUnfAdjoint: k_adjoint<R><<<per_w, kBlock, 0, s>>>(a); break;
    case kUnfU: k_u<R><<<per_atom, kBlock, 0, s>>>(a); break;
    case kUnfV: k_v<R><<<per_atom, kBlock, 0, s>>>(a); break;
    case kUnfForce: k_force<R><<<per_atom, kBlock, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_unfused(int stage, int precision, const UnfusedArgs& a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  // grids are sized in 32 bits: one work-group per four atoms or per 256
  // entries or elements
  if (a.n * D * K / kBlock >= (1LL << 31) || a.n_entries / kBlock >= (1LL << 31)) return hipErrorInvalidValue;
  if (precision == 64) return launch_stage<double>(stage, a, s);
  if (precision == 32) return launch_stage<float>(stage, a, s);
  return hipErrorInvalidValue;
}

}  // namespace mlip
