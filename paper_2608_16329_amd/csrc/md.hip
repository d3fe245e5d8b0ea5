// Velocity-Verlet driver kernels (metal units).  Not part of the potential:
// they move atoms between force evaluations, as the MD code around the MLIP
// does in the paper's LAMMPS runs (Section 4.1).
#include "mlip_internal.h"

namespace mlip {
namespace {

__device__ inline void atomic_max_nonneg(double* addr, double v) {
  // non-negative doubles order like their bit patterns
  atomicMax(reinterpret_cast<unsigned long long*>(addr), static_cast<unsigned long long>(__double_as_longlong(v)));
}

__global__ void k_first_half(double* __restrict__ pos, double* __restrict__ vel, const double* __restrict__ f,
                             const int32_t* __restrict__ types, const double* __restrict__ inv_mass, int64_t n,
                             double dt, const double* __restrict__ ref, double* __restrict__ max_disp2) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  double d2 = 0.0;
  if (i < n) {
    const double s = 0.5 * dt * inv_mass[types[i]];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      const double v = vel[3 * i + k] + s * f[3 * i + k];
      vel[3 * i + k] = v;
      const double x = pos[3 * i + k] + dt * v;
      pos[3 * i + k] = x;
      if (ref) {
        const double d = x - ref[3 * i + k];
        d2 += d * d;
      }
    }
  }
  if (ref) {
    for (int o = 32; o > 0; o >>= 1) d2 = fmax(d2, __shfl_xor(d2, o, 64));
    if ((threadIdx.x & 63) == 0) atomic_max_nonneg(max_disp2, d2);
  }
}

__global__ void k_second_half(double* __restrict__ vel, const double* __restrict__ f,
                              const int32_t* __restrict__ types, const double* __restrict__ inv_mass, int64_t n,
                              double dt) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const double s = 0.5 * dt * inv_mass[types[i]];
#pragma unroll
  for (int k = 0; k < 3; ++k) vel[3 * i + k] += s * f[3 * i + k];
}

// largest squared displacement since the last neighbour build, against the
// wrapped build-time positions kept in sorted order (minimum image)
__global__ void k_disp_since_build(const double* __restrict__ pos, const int32_t* __restrict__ perm,
                                   const double* __restrict__ spos, int64_t n, double bx, double by, double bz,
                                   double* __restrict__ max_disp2) {
  const int64_t a = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  double d2 = 0.0;
  if (a < n) {
    const int64_t i = perm[a];
    double dx = pos[3 * i] - spos[3 * a], dy = pos[3 * i + 1] - spos[3 * a + 1], dz = pos[3 * i + 2] - spos[3 * a + 2];
    dx -= bx * rint(dx / bx);
    dy -= by * rint(dy / by);
    dz -= bz * rint(dz / bz);
    d2 = dx * dx + dy * dy + dz * dz;
  }
  for (int o = 32; o > 0; o >>= 1) d2 = fmax(d2, __shfl_xor(d2, o, 64));
  if ((threadIdx.x & 63) == 0) atomic_max_nonneg(max_disp2, d2);
}

// sum m v^2 / 2 in eV: inv_mass holds acc/m, so m = acc / inv_mass
__global__ void k_kinetic(const double* __restrict__ vel, const int32_t* __restrict__ types,
                          const double* __restrict__ inv_mass, int64_t n, double* __restrict__ out) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  double e = 0.0;
  if (i < n) {
    const double v2 = vel[3 * i] * vel[3 * i] + vel[3 * i + 1] * vel[3 * i + 1] + vel[3 * i + 2] * vel[3 * i + 2];
    e = 0.5 * v2 / inv_mass[types[i]];
  }
  for (int o = 32; o > 0; o >>= 1) e += __shfl_xor(e, o, 64);
  if ((threadIdx.x & 63) == 0) atomicAdd(out, e);
}

inline unsigned blocks_for(int64_t n) { return unsigned((n + 255) / 256); }

}  // namespace

hipError_t launch_md_first_half(double* pos, double* vel, const double* forces, const int32_t* types,
                                const double* inv_mass, int64_t n, double dt, const double* ref,
                                double* max_disp2, hipStream_t s) {
  k_first_half<<<blocks_for(n), 256, 0, s>>>(pos, vel, forces, types, inv_mass, n, dt, ref, max_disp2);
  return hipGetLastError();
}

hipError_t launch_md_disp_since_build(const double* pos, const int32_t* perm, const double* spos, int64_t n,
                                     const double box[3], double* max_disp2, hipStream_t s) {
  k_disp_since_build<<<blocks_for(n), 256, 0, s>>>(pos, perm, spos, n, box[0], box[1], box[2], max_disp2);
  return hipGetLastError();
}

hipError_t launch_md_second_half(double* vel, const double* forces, const int32_t* types,
                                 const double* inv_mass, int64_t n, double dt, hipStream_t s) {
  k_second_half<<<blocks_for(n), 256, 0, s>>>(vel, forces, types, inv_mass, n, dt);
  return hipGetLastError();
}

hipError_t launch_md_kinetic(const double* vel, const int32_t* types, const double* inv_mass, int64_t n,
                             double* out, hipStream_t s) {
  k_kinetic<<<blocks_for(n), 256, 0, s>>>(vel, types, inv_mass, n, out);
  return hipGetLastError();
}

}  // namespace mlip
