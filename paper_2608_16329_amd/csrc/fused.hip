// Fused energy / force / virial kernel for gfx950 (Section 3.1, Eqs. 1-10;
// fusion as in Section 3.4, re-designed for CDNA4).
//
// One persistent work-group (4 wavefronts, one per SIMD) walks a list of
// tiles.  A tile is up to 16 centre atoms of one species, consecutive in the
// cell-sorted order.  Per tile:
//
//   A. Stage the tile's atoms and neighbour rows; keep pairs with r < r_c and
//      bucket them by neighbour species in LDS, in atom order.  Each bucket
//      is cut into 16-pair chunks; all pairs of a chunk share one encoder
//      table (pair conditioning, Section 3.2).
//   B. Pass 1, one chunk per wavefront at a time: the radial encoder (Eq. 2)
//      and its derivative in r run as MFMA 16x16x4 products with the
//      16 pairs as one matrix dimension, the activation and its tangent
//      stacked as two column tiles sharing every weight fragment.  The
//      moment P_i = sum_j g_ang (x) g_rad (Eq. 4) is another MFMA product
//      (K = pairs), accumulated into LDS.  The pre-cutoff output m and its
//      tangent dm (2k values per pair) go to a fixed-size per-work-group
//      workspace; nothing is recomputed in pass 2.  When the encoder is
//      recomputed in pass 2 instead (no workspace), pass 1 runs the forward
//      products alone: the moment needs m only.
//   C. Descriptor (Eq. 5), energy head (Eq. 6) and its gradient, and
//      W_i = dE_i/dP_i (Eq. 7) for the tile's atoms, in LDS (W overwrites P).
//   D. Pass 2, per chunk: v = W g and the reassociated radial term
//      s = g_ang^T W g' (Eqs. 8-9; U_i is never formed) as MFMA products,
//      then f_ij (Eq. 10), scatter F_j -= f_ij (global atomics) and
//      F_i += f_ij, w_i -= r_ij (x) f_ij (LDS atomics).
//   E. Write E_i, w_i, add F_i; block-reduce totals.
//
// The kernel is instantiated for two arithmetic types R of the network and
// the contractions: float64 (the paper's evaluation precision, Section 4.1)
// and float32 (the reduced-precision mode evaluated beside it, Sections 3.4
// and 4.4).  The minimum-image difference of positions and every output
// accumulation (F_i, F_j, w_i, E, totals) stay in float64 in both; r, the
// unit vector, the cutoff function, the network, the angular features, the
// moment, W, the two pass-2 contractions and the partial force use R.
//
// MFMA 16x16x4 register layout on gfx950 (lane = 16*g + c), for both types:
//   A operand: lane holds A[c][g]; B operand: lane holds B[g][c].
// The result layout differs: register q of lane holds D[drow(q, g)][c] with
// drow = 4q + g for float64 and 4g + q for float32.  A D-tile X can feed a
// later product as B (contracting over its rows; k-step q covers rows
// drow(q, 0..3)) or as A (X^T, same contraction); the host packs weight
// fragments with the same row map.
#include "kernel_math.h"
#include "mlip_internal.h"

namespace mlip {
namespace {

typedef double v4d __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

template <typename R>
struct Vec4;
template <>
struct Vec4<double> {
  typedef v4d type;
};
template <>
struct Vec4<float> {
  typedef v4f type;
};
template <typename R>
using v4 = typename Vec4<R>::type;

__device__ __forceinline__ v4d mfma(double a, double b, v4d c) {
  return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ v4f mfma(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Result row held in register q of a lane of group g, and its inverse: row c
// sits in register qof(c) of the lanes of group gof(c).
template <typename R>
__device__ __forceinline__ int drow(int q, int g) {
  return sizeof(R) == 8 ? 4 * q + g : 4 * g + q;
}
template <typename R>
__device__ __forceinline__ int qof(int c) {
  return sizeof(R) == 8 ? c >> 2 : c & 3;
}
template <typename R>
__device__ __forceinline__ int gof(int c) {
  return sizeof(R) == 8 ? c & 3 : c >> 2;
}

// Logistic sigmoid 1 / (1 + exp(-z)) in float64, written out so the VALU
// cost stays low next to the MFMA work (on gfx950 float64 VALU instructions
// and float64 MFMA share one pipe, so every instruction here delays the
// matrix products):
//  * exp(t), t = -z clamped to [-700, 700] (beyond that the sigmoid is 0 or 1
//    to far below float64 resolution of the SiLU value), by Cody-Waite
//    reduction t = n ln2 + r with |r| <= ln2/2, a degree-10 polynomial (the
//    interpolant at Chebyshev nodes, below 3.4e-16 relative error) and a 2^n
//    scaling;
//  * 1 / (1 + e) from the hardware reciprocal estimate (relative error
//    measured below 2^-24) refined by one Newton-Raphson step, which squares
//    that error.
__device__ __forceinline__ double sigmoid(double z) {
  constexpr double kLog2e = 1.4426950408889634;
  constexpr double kLn2Hi = 6.93147180369123816490e-01;  // ln2 split, high part exact in 32 bits
  constexpr double kLn2Lo = 1.90821492927058770002e-10;
  const double t = fmin(fmax(-z, -700.0), 700.0);
  const double n = rint(t * kLog2e);
  double r = fma(-n, kLn2Hi, t);
  r = fma(-n, kLn2Lo, r);
  // polynomial interpolating exp at the 11 Chebyshev nodes of [-ln2/2,
  // ln2/2] (solved in 80-bit arithmetic, rounded to float64), highest power
  // first; relative error below 3.4e-16 on the interval
  constexpr double c[11] = {
    2.762635356445665e-07,  2.764018186396873e-06, 2.4801504368699663e-05, 0.00019841170267682938,
    0.0013888888932453442,  0.008333333385670185,  0.04166666666657336,    0.16666666666554397,
    0.5000000000000006,     1.0000000000000067,    1.0};
  double p = c[0];
#pragma unroll
  for (int k = 1; k < 11; ++k) p = fma(p, r, c[k]);
  const double d = 1.0 + ldexp(p, int(n));
  const double y = __builtin_amdgcn_rcp(d);
  return fma(fma(-d, y, 1.0), y, y);
}

// Logistic sigmoid in float32 from the hardware base-2 exponential and
// reciprocal (each within about one ulp).  For large -z the exponential
// overflows to +inf and the reciprocal returns 0, the sigmoid's limit; for
// large z it underflows to 0 and the result is 1.
__device__ __forceinline__ float sigmoid(float z) {
  constexpr float kLog2e = 1.44269504f;
  const float e = __builtin_amdgcn_exp2f(-z * kLog2e);
  return __builtin_amdgcn_rcpf(1.0f + e);
}

// Slope of the SiLU z s(z), s (1 + z (1 - s)), as two fused multiply-adds:
// t = z - s z = z (1 - s), then s + s t.
template <typename R>
__device__ __forceinline__ R silu_slope(R z, R s) {
  return fma(s, fma(-s, z, z), s);
}

// Pair geometry after the minimum-image difference (which stays in float64):
// IEEE float64 square root and division, or the float32 hardware
// instructions (about one ulp).
__device__ __forceinline__ double vsqrt(double x) { return sqrt(x); }
__device__ __forceinline__ float vsqrt(float x) { return __builtin_amdgcn_sqrtf(x); }
__device__ __forceinline__ double vrcp(double x) { return 1.0 / x; }
__device__ __forceinline__ float vrcp(float x) { return __builtin_amdgcn_rcpf(x); }

// cos(x) and sin(x) for 0 <= x < pi (the cutoff function's argument, x =
// pi r / r_c with r < r_c) in float64: Cody-Waite reduction x = k pi/2 + y
// with k = rint(2x / pi) in {0, 1, 2} and |y| <= pi/4, the Taylor
// polynomials of sin (degree 15) and cos (degree 16) in y (truncation below
// 5e-17 and 3e-18; at degrees 13 and 14 the 2e-14 error of fc reached 6e-10
// in the forces of deep networks), then the quadrant rotation.  The general
// library routines carry range reduction for any argument, which this path
// never needs.
__device__ __forceinline__ void cut_sincos(double x, double* sn, double* cs) {
  constexpr double kTwoOverPi = 0.63661977236758134308;
  constexpr double kPio2Hi = 1.57079632679489655800e+00;  // pi/2 = hi + lo
  constexpr double kPio2Lo = 6.12323399573676603587e-17;
  const double k = rint(x * kTwoOverPi);
  double y = fma(-k, kPio2Hi, x);
  y = fma(-k, kPio2Lo, y);
  const double y2 = y * y;
  // 1 / n! for the odd (sin) and even (cos) terms, highest first
  double ps = -7.647163731819816e-13;  // -1/15!
  ps = fma(ps, y2, 1.6059043836821613e-10);  // 1/13!
  ps = fma(ps, y2, -2.505210838544172e-08);  // -1/11!
  ps = fma(ps, y2, 2.7557319223985893e-06);  // 1/9!
  ps = fma(ps, y2, -1.984126984126984e-04);  // -1/7!
  ps = fma(ps, y2, 8.333333333333333e-03);   // 1/5!
  ps = fma(ps, y2, -1.6666666666666666e-01); // -1/3!
  const double sy = fma(ps * y2, y, y);
  double pc = 4.779477332387385e-14;  // 1/16!
  pc = fma(pc, y2, -1.1470745597729725e-11); // -1/14!
  pc = fma(pc, y2, 2.08767569878681e-09);    // 1/12!
  pc = fma(pc, y2, -2.755731922398589e-07);  // -1/10!
  pc = fma(pc, y2, 2.48015873015873e-05);    // 1/8!
  pc = fma(pc, y2, -1.388888888888889e-03);  // -1/6!
  pc = fma(pc, y2, 4.1666666666666664e-02);  // 1/4!
  pc = fma(pc, y2, -0.5);                    // -1/2!
  const double cy = fma(pc, y2, 1.0);
  const int q = int(k);
  *sn = q == 0 ? sy : (q == 1 ? cy : -sy);
  *cs = q == 0 ? cy : (q == 1 ? -sy : -cy);
}

// Cutoff function fc(r) = (1 + cos(pi r / r_c)) / 2 and its derivative
// -(pi / r_c) sin(pi r / r_c) / 2 for r < r_c (Eq. 2): float64 from the
// reduced-range routine above, float32 from the hardware sine and cosine
// (about one ulp; they take revolutions).
__device__ __forceinline__ void cutoff(double r, double pi_rc, double* fc, double* dfc) {
  double sn, cs;
  cut_sincos(r * pi_rc, &sn, &cs);
  *fc = 0.5 * (1.0 + cs);
  *dfc = -0.5 * pi_rc * sn;
}
__device__ __forceinline__ void cutoff(float r, float pi_rc, float* fc, float* dfc) {
  const float x = r * pi_rc * 0.159154943f;
  *fc = 0.5f * (1.0f + __builtin_amdgcn_cosf(x));
  *dfc = -0.5f * pi_rc * __builtin_amdgcn_sinf(x);
}

// Exponents (a, b, c) of the Cartesian monomials of degree <= 5, degree by
// degree and lexicographic with x first within a degree (the column order of
// the angular table; its first 20 entries are the order of `monomials`).
struct MonoExp {
  unsigned char e[56][3];
  constexpr MonoExp() : e{} {
    int i = 0;
    for (int d = 0; d <= 5; ++d)
      for (int a = d; a >= 0; --a)
        for (int b = d - a; b >= 0; --b) {
          e[i][0] = (unsigned char)a;
          e[i][1] = (unsigned char)b;
          e[i][2] = (unsigned char)(d - a - b);
          ++i;
        }
  }
};
constexpr MonoExp kMonoExp{};

// The NM monomials (20: degree <= 3, 56: degree <= 5) of (x, y, z) and, when
// kGrad, their gradients.
template <int NM, bool kGrad, typename R>
__device__ __forceinline__ void monomials_n(R x, R y, R z, R m[NM], R gx[NM], R gy[NM], R gz[NM]) {
  if constexpr (NM == kMonomials) {
    monomials(x, y, z, m);
    if (kGrad) monomial_grads(x, y, z, gx, gy, gz);
  } else {
    R px[6], py[6], pz[6];
    px[0] = py[0] = pz[0] = R(1);
#pragma unroll
    for (int k = 1; k < 6; ++k) {
      px[k] = px[k - 1] * x;
      py[k] = py[k - 1] * y;
      pz[k] = pz[k - 1] * z;
    }
#pragma unroll
    for (int i = 0; i < NM; ++i) {
      const int a = kMonoExp.e[i][0], b = kMonoExp.e[i][1], c = kMonoExp.e[i][2];
      m[i] = px[a] * py[b] * pz[c];
      if (kGrad) {
        gx[i] = a ? R(a) * px[a > 0 ? a - 1 : 0] * py[b] * pz[c] : R(0);
        gy[i] = b ? R(b) * px[a] * py[b > 0 ? b - 1 : 0] * pz[c] : R(0);
        gz[i] = c ? R(c) * px[a] * py[b] * pz[c > 0 ? c - 1 : 0] : R(0);
      }
    }
  }
}

// Slots of the per-tile table of the tile-reduced force scatter: a tile of
// up to 32 atoms has a few hundred distinct neighbours.
constexpr int kFjSlots = 1024;

// Rows of the moment kept in LDS: the angular rows of the configuration (16
// irreducible rows to l_max 3, the Cartesian basis's 20, 36 to l_max 5) of
// the DR rows that its 16-row MFMA tiles span; the rows past them are zero
// in every product and are neither stored nor read.
constexpr int moment_rows(int DR, int NM) { return NM == 56 ? 36 : (DR == 32 ? 20 : DR); }

template <int K, int TM, typename R, int NW, int DR, int NM>
struct Smem {
  R P[TM][moment_rows(DR, NM)][K + 1];  // moment, then its adjoint W (padded columns)
  // Pass 1 reads the first-layer weights; the head runs after pass 1 and
  // before the next tile is staged, so its activations reuse those bytes.
  union {
    R l0[kMaxSpecies][2][kEncWidth];  // w0, b0 of the tile's encoder tables, by neighbour species
    struct {
      R xT[(NM == 20 ? 4 : 6) * K][TM > 16 ? 32 : 16];  // head input vec(G), feature-major
      R yT[kHeadWidth][TM > 16 ? 32 : 16];             // head activations
      R gT[kHeadWidth][TM > 16 ? 32 : 16];             // head backward scratch
    } hd;
    // pass 2 of the cached configuration with the tile-reduced force
    // scatter: the tile's F_j contributions summed per neighbour j
    struct {
      int key[kFjSlots];        // neighbour index, -1 = empty
      double val[kFjSlots][3];
    } fj;
  } u;
  R qc[DR][NM];        // angular features over the monomials
  R rw[DR];            // descriptor weight of each angular row (metric C_l)
  double tpos[TM][3];
  double Fi[TM][3];
  double Wi[TM][9];
  double Ei[TM];
  long long row_beg[TM];
  int ent_base[TM + 1];
  int orig[TM];
  int cand[TM][9];     // cells scanned around each atom's cell (decoding coded list entries)
  int cnt[kMaxSpecies][TM];
  int base[kMaxSpecies][TM];
  int pair_j[tile_entry_cap(TM)];
  unsigned char pair_a[tile_entry_cap(TM)];
  int wsum[NW];
  int a0;
  int ch_start[tile_chunk_cap(TM)];
  unsigned char ch_count[tile_chunk_cap(TM)];
  unsigned char ch_s[tile_chunk_cap(TM)];
  int n_chunks;
  int next_chunk[2];  // dynamic chunk hand-out of pass 1 and pass 2
  int n_active;
  int tile_species;
  int na;
};

// Position of the neighbour in column c of chunk ch (or a dummy), fetched
// one chunk ahead so its latency overlaps the previous chunk's work.
struct PairPos {
  double x, y, z;
};

// Value of group g (0..3) among four, by bit masks: a select chain on the
// lane-dependent g would otherwise be compiled into divergent branches.
__device__ __forceinline__ double pick4(int g, double m0, double m1, double m2, double m3) {
  const unsigned long long s1 = 0ull - (unsigned long long)(g & 1), s2 = 0ull - (unsigned long long)((g >> 1) & 1);
  const unsigned long long lo = (__double_as_longlong(m0) & ~s1) | (__double_as_longlong(m1) & s1);
  const unsigned long long hi = (__double_as_longlong(m2) & ~s1) | (__double_as_longlong(m3) & s1);
  return __longlong_as_double((long long)((lo & ~s2) | (hi & s2)));
}
__device__ __forceinline__ float pick4(int g, float m0, float m1, float m2, float m3) {
  const unsigned s1 = 0u - unsigned(g & 1), s2 = 0u - unsigned((g >> 1) & 1);
  const unsigned lo = (__float_as_uint(m0) & ~s1) | (__float_as_uint(m1) & s1);
  const unsigned hi = (__float_as_uint(m2) & ~s1) | (__float_as_uint(m3) & s1);
  return __uint_as_float((lo & ~s2) | (hi & s2));
}

// Next chunk for this wavefront: chunks are handed out in order from an LDS
// counter, so a wavefront that runs ahead of its SIMD partner takes more of
// them and the wavefronts of a tile finish together.
__device__ __forceinline__ int grab_chunk(int* counter) {
  int v = 0;
  if ((threadIdx.x & 63) == 0) v = atomicAdd(counter, 1);
  return __builtin_amdgcn_readfirstlane(__shfl(v, 0, 64));
}

template <int K, int TM, typename R, int NW, int DR, int NM>
__device__ __forceinline__ PairPos load_pair_pos(const FusedArgs& A, const Smem<K, TM, R, NW, DR, NM>& S, int ch) {
  const int c = threadIdx.x & 15;
  PairPos p{0.0, 0.0, 0.0};
  if (c < S.ch_count[ch]) {
    const long long j = S.pair_j[S.ch_start[ch] + c];
    p.x = A.pos[3 * j];
    p.y = A.pos[3 * j + 1];
    p.z = A.pos[3 * j + 2];
  }
  return p;
}

// Weight-fragment streaming of the encoder products: fragments of VW
// consecutive output tiles per 16-byte load, through register rings issued
// kRing - 1 (hidden layers) or kRingO - 1 (output layer) k-steps ahead of the
// MFMAs that consume them.  An output-layer k-step is only 2 KT products, so
// its ring runs further ahead.  The float32 kernel runs two wavefronts per
// SIMD, which cover each other's load latency; there shallower rings leave
// more registers and measured faster (ring depths 2 and 4 against 3 and 8).
// Fragment array at a wave-uniform address, read through a buffer descriptor:
// the descriptor and each group's offset are scalar and the lane offset is
// one fixed vector register, so walking the array costs no vector address
// arithmetic (which on this part would share the pipe with the float64
// MFMAs); a read past `bytes` returns zero instead of touching other memory.
// Group e holds one V per lane, lane l at byte (64 e + l) sizeof(V).
constexpr int kRawBufferConfig = 0x00020000;  // raw untyped access, gfx9-family descriptor word 3
template <typename V>
struct FragStream {
  __amdgpu_buffer_rsrc_t rs;
  int lo;
  __device__ __forceinline__ FragStream(const void* base, int bytes)
      : rs(__builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, kRawBufferConfig)),
        lo(int(threadIdx.x & 63) * int(sizeof(V))) {}
  __device__ __forceinline__ V operator[](int e) const {
    const int so = e * 64 * int(sizeof(V));
    if constexpr (sizeof(V) == 16) return __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b128(rs, lo, so, 0));
    else if constexpr (sizeof(V) == 8) return __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b64(rs, lo, so, 0));
    else return __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b32(rs, lo, so, 0));
  }
};

// Bias vector of a hidden layer at a wave-uniform address, read through a
// buffer descriptor in the accumulator row order: element (To, q) of lane
// (g, c) is row 16 To + drow(q, g); the lane part of that offset is one
// fixed vector register, the rest a scalar offset.  With bytes = 0 every
// read returns zero without touching memory.
template <typename R>
struct BiasStream {
  __amdgpu_buffer_rsrc_t rs;
  int lo;
  __device__ __forceinline__ BiasStream(const void* base, int bytes, int g)
      : rs(__builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, kRawBufferConfig)),
        lo((sizeof(R) == 8 ? g : 4 * g) * int(sizeof(R))) {}
  __device__ __forceinline__ R operator()(int To, int q) const {
    const int so = (16 * To + (sizeof(R) == 8 ? 4 * q : q)) * int(sizeof(R));
    if constexpr (sizeof(R) == 8) return __builtin_bit_cast(R, __builtin_amdgcn_raw_buffer_load_b64(rs, lo, so, 0));
    else return __builtin_bit_cast(R, __builtin_amdgcn_raw_buffer_load_b32(rs, lo, so, 0));
  }
};

template <int K, typename R>
struct Stream {
  static constexpr int KT = K / 16;
  static constexpr int VW = 16 / int(sizeof(R));  // fragments per load
  static constexpr int NH = 8 / VW;               // loads per hidden-layer k-step
  static constexpr int VO = KT < VW ? KT : VW;    // fragments per output-layer load
  static constexpr int NO = KT / VO;              // loads per output-layer k-step
  static constexpr int kRing = sizeof(R) == 8 ? 3 : 2;
  static constexpr int kRingO = sizeof(R) == 8 ? 8 : 4;
  typedef R vh_t __attribute__((ext_vector_type(VW)));
  typedef R vo_t __attribute__((ext_vector_type(VO)));
};

// Minimum-image vector r_ij of the pair in column c of chunk ch (Eq. 1), in
// float64; (1, 0, 0) and atom -1 for the padding columns of a partial chunk.
template <int K, int TM, typename R, int NW, int DR, int NM>
__device__ __forceinline__ void pair_delta(const FusedArgs& A, const Smem<K, TM, R, NW, DR, NM>& S, int ch,
                                           const PairPos& pp, double* dx, double* dy, double* dz, int* atom) {
  const int c = threadIdx.x & 15;
  *dx = 1.0; *dy = 0.0; *dz = 0.0; *atom = -1;
  if (c >= S.ch_count[ch]) return;
  const int a = S.pair_a[S.ch_start[ch] + c];
  *dx = fold(pp.x - S.tpos[a][0], A.box[0], A.inv_box[0]);
  *dy = fold(pp.y - S.tpos[a][1], A.box[1], A.inv_box[1]);
  *dz = fold(pp.z - S.tpos[a][2], A.box[2], A.inv_box[2]);
  *atom = a;
}

// Encoder table of chunk ch (pair conditioning, Section 3.2).
template <int K, int TM, typename R, int NW, int DR, int NM>
__device__ __forceinline__ const R* chunk_table(const FusedArgs& A, const Smem<K, TM, R, NW, DR, NM>& S, int ch) {
  // the same for every lane: kept in scalar registers, so the weight loads
  // take a scalar base and the k-step offsets cost no vector instructions
  const int sj = __builtin_amdgcn_readfirstlane(S.ch_s[ch]);
  const int si = __builtin_amdgcn_readfirstlane(S.tile_species);
  const int tau = A.enc_cond == 2 ? si * A.C + sj : (A.enc_cond == 1 ? sj : 0);
  return static_cast<const R*>(A.enc) + (long long)tau * A.enc_stride;
}

// Encoder forward and tangent (Eq. 2 and its derivative in r) up to the last
// hidden layer for the 16 pairs of a chunk: the first layer (scalar input)
// from the LDS copy of (w0, b0), then the residual hidden layers Z = W H as
// 8 x 32 MFMA steps whose forward and tangent columns share each weight
// fragment.  On return h[T][i], dh[T][i] hold rows 16T + drow(i, g) of
// column c; the result is the output-layer section of the table.  Without
// kTan only the forward runs (dh is left untouched): the moment needs the
// encoder output alone, so a pass 1 that keeps no workspace skips the
// tangent's half of the products.
template <int K, int TM, typename R, int NW, int DR, int NM, bool kTan = true>
__device__ __forceinline__ const R* encoder_hidden(const FusedArgs& A, const Smem<K, TM, R, NW, DR, NM>& S, int sj, R r,
                                                   const R* __restrict__ tab, R (&h)[8][4], R (&dh)[8][4]) {
  typedef Stream<K, R> St;
  typedef typename St::vh_t vh_t;
  constexpr int NH = St::NH, VW = St::VW, kRing = St::kRing;
  const int lane = threadIdx.x & 63, g = lane >> 4;
  constexpr int kLayerBytes = int(kEncWidth * kEncWidth * sizeof(R));
  constexpr int kBiasBytes = int(kEncWidth * sizeof(R));
  const int nh = A.enc_hidden;
  // The first hidden layer's leading weight fragments are requested before
  // the elementwise first layer, whose activation work covers their
  // latency; each hidden layer requests the next one's in its last k-steps,
  // so they arrive during its own activation phase.  Past the last hidden
  // layer that descriptor has size 0 and reads zeros.  At k = 64 the wider
  // output tiles leave no registers for fragments held across an activation
  // phase (it measured slower): there each layer fills its ring at its start.
  constexpr bool kCross = K <= 32;
  const R* __restrict__ layer = tab + 2 * kEncWidth;
  vh_t wb[kRing][NH];
  v4<R> acc[8], dacc[8];
  if constexpr (kCross) {
    const FragStream<vh_t> frag(layer, nh > 1 ? kLayerBytes : 0);
#pragma unroll
    for (int p = 0; p < kRing - 1; ++p)
#pragma unroll
      for (int u = 0; u < NH; ++u) wb[p][u] = frag[p * NH + u];
  }
#pragma unroll
  for (int T = 0; T < 8; ++T)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int in = 16 * T + drow<R>(i, g);
      const R w0 = S.u.l0[sj][0][in], z = w0 * r + S.u.l0[sj][1][in];
      const R s = sigmoid(z);
      h[T][i] = z * s;
      if constexpr (kTan) dh[T][i] = silu_slope(z, s) * w0;
    }
  for (int t = 1; t < nh; ++t) {
    const FragStream<vh_t> frag(layer, kLayerBytes);
    const R* __restrict__ next = layer + kEncWidth * kEncWidth + kEncWidth;
    const bool more = t + 1 < nh;
    const FragStream<vh_t> nfrag(next, more ? kLayerBytes : 0);
    if constexpr (!kCross) {
#pragma unroll
      for (int p = 0; p < kRing - 1; ++p)
#pragma unroll
        for (int u = 0; u < NH; ++u) wb[p][u] = frag[p * NH + u];
    }
    // the tangent has no bias
    {
      const BiasStream<R> bias(layer + kEncWidth * kEncWidth, kBiasBytes, g);
#pragma unroll
      for (int To = 0; To < 8; ++To) acc[To] = v4<R>{bias(To, 0), bias(To, 1), bias(To, 2), bias(To, 3)};
    }
#pragma unroll
    for (int To = 0; To < 8; ++To) dacc[To] = v4<R>{0, 0, 0, 0};
#pragma unroll
    for (int ks = 0; ks < 32; ++ks) {
      const int kn = ks + kRing - 1;
      if (kCross || kn < 32) {
#pragma unroll
        for (int u = 0; u < NH; ++u) wb[kn % kRing][u] = kn < 32 ? frag[kn * NH + u] : nfrag[(kn - 32) * NH + u];
      }
      __builtin_amdgcn_sched_barrier(0);
      const int T = ks >> 2, i = ks & 3;
#pragma unroll
      for (int To = 0; To < 8; ++To) {
        const R wv = wb[ks % kRing][To / VW][To % VW];
        acc[To] = mfma(wv, h[T][i], acc[To]);
        if constexpr (kTan) dacc[To] = mfma(wv, dh[T][i], dacc[To]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    // the next layer's k-step p sits in slot (32 + p) mod kRing; it starts
    // from slot p (a no-op when kRing divides 32)
    if constexpr (kCross && 32 % kRing != 0) {
      vh_t nx[kRing - 1][NH];
#pragma unroll
      for (int p = 0; p < kRing - 1; ++p)
#pragma unroll
        for (int u = 0; u < NH; ++u) nx[p][u] = wb[(32 + p) % kRing][u];
#pragma unroll
      for (int p = 0; p < kRing - 1; ++p)
#pragma unroll
        for (int u = 0; u < NH; ++u) wb[p][u] = nx[p][u];
    }
#pragma unroll
    for (int To = 0; To < 8; ++To) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const R z = acc[To][q];
        const R s = sigmoid(z);
        h[To][q] += z * s;
        if constexpr (kTan) dh[To][q] = fma(silu_slope(z, s), dacc[To][q], dh[To][q]);
      }
    }
    layer = next;
  }
  return layer;
}

// Encoder output layer with pairs as rows: mo[Tc] register q holds
// m[pair drow(q, g)][16Tc + c] (dmo the same for the tangent, computed only
// with kTan).  Even and odd k-steps accumulate separately so 4 KT independent
// MFMA chains are in flight; the bias is added at the end so the first
// products do not wait for its load.
template <int K, typename R, bool kTan = true>
__device__ __forceinline__ void encoder_out_rows(const R* __restrict__ layer, const R (&h)[8][4], const R (&dh)[8][4],
                                                 v4<R> (&mo)[K / 16], v4<R> (&dmo)[K / 16]) {
  typedef Stream<K, R> St;
  typedef typename St::vo_t vo_t;
  constexpr int KT = St::KT, NO = St::NO, VO = St::VO, kRing = St::kRingO;
  const int lane = threadIdx.x & 63, c = lane & 15;
  const R* __restrict__ bout = layer + K * kEncWidth;
  v4<R> mo2[2][KT], dmo2[2][KT];
  R b[KT];
#pragma unroll
  for (int Tc = 0; Tc < KT; ++Tc) {
    b[Tc] = bout[16 * Tc + c];
    mo2[0][Tc] = mo2[1][Tc] = dmo2[0][Tc] = dmo2[1][Tc] = v4<R>{0, 0, 0, 0};
  }
  const FragStream<vo_t> frag(layer, int(K * kEncWidth * sizeof(R)));
  vo_t wo[kRing][NO];
#pragma unroll
  for (int p = 0; p < kRing - 1; ++p)
#pragma unroll
    for (int u = 0; u < NO; ++u) wo[p][u] = frag[p * NO + u];
#pragma unroll
  for (int ks = 0; ks < 32; ++ks) {
    if (ks + kRing - 1 < 32) {
#pragma unroll
      for (int u = 0; u < NO; ++u) wo[(ks + kRing - 1) % kRing][u] = frag[(ks + kRing - 1) * NO + u];
    }
    __builtin_amdgcn_sched_barrier(0);
    const int T = ks >> 2, i = ks & 3;
#pragma unroll
    for (int Tc = 0; Tc < KT; ++Tc) {
      const R wv = wo[ks % kRing][Tc / VO][Tc % VO];
      mo2[ks & 1][Tc] = mfma(h[T][i], wv, mo2[ks & 1][Tc]);
      if constexpr (kTan) dmo2[ks & 1][Tc] = mfma(dh[T][i], wv, dmo2[ks & 1][Tc]);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int Tc = 0; Tc < KT; ++Tc) {
    mo[Tc] = mo2[0][Tc] + mo2[1][Tc] + v4<R>{b[Tc], b[Tc], b[Tc], b[Tc]};
    if constexpr (kTan) dmo[Tc] = dmo2[0][Tc] + dmo2[1][Tc];
  }
}

// Encoder output layer with pairs as columns (the same fragments serve as
// the A operand): register q of lane (g, c) for output tile Tc holds
// m[pair c][16Tc + drow(q, g)], which is exactly the B operand of pass 2's
// W m product.
template <int K, typename R>
__device__ __forceinline__ void encoder_out_cols(const R* __restrict__ layer, const R (&h)[8][4], const R (&dh)[8][4],
                                                 R (&mB)[K / 16][4], R (&dmB)[K / 16][4]) {
  typedef Stream<K, R> St;
  typedef typename St::vo_t vo_t;
  constexpr int KT = St::KT, NO = St::NO, VO = St::VO, kRing = St::kRingO;
  const int lane = threadIdx.x & 63, g = lane >> 4;
  const R* __restrict__ bout = layer + K * kEncWidth;
  v4<R> acc[KT], dacc[KT];
#pragma unroll
  for (int Tc = 0; Tc < KT; ++Tc) {
    acc[Tc] = v4<R>{bout[16 * Tc + drow<R>(0, g)], bout[16 * Tc + drow<R>(1, g)], bout[16 * Tc + drow<R>(2, g)],
                    bout[16 * Tc + drow<R>(3, g)]};
    dacc[Tc] = v4<R>{0, 0, 0, 0};
  }
  const FragStream<vo_t> frag(layer, int(K * kEncWidth * sizeof(R)));
  vo_t wo[kRing][NO];
#pragma unroll
  for (int p = 0; p < kRing - 1; ++p)
#pragma unroll
    for (int u = 0; u < NO; ++u) wo[p][u] = frag[p * NO + u];
#pragma unroll
  for (int ks = 0; ks < 32; ++ks) {
    if (ks + kRing - 1 < 32) {
#pragma unroll
      for (int u = 0; u < NO; ++u) wo[(ks + kRing - 1) % kRing][u] = frag[(ks + kRing - 1) * NO + u];
    }
    __builtin_amdgcn_sched_barrier(0);
    const int T = ks >> 2, i = ks & 3;
#pragma unroll
    for (int Tc = 0; Tc < KT; ++Tc) {
      const R wv = wo[ks % kRing][Tc / VO][Tc % VO];
      acc[Tc] = mfma(wv, h[T][i], acc[Tc]);
      dacc[Tc] = mfma(wv, dh[T][i], dacc[Tc]);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int Tc = 0; Tc < KT; ++Tc)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      mB[Tc][q] = acc[Tc][q];
      dmB[Tc][q] = dacc[Tc][q];
    }
}

// Pass 1 on one chunk: encoder forward, moment accumulation and, when kWs,
// the encoder tangent and the workspace write of (m, dm).
template <int K, int TM, typename R, int NW, int DR, int NM, bool kWs>
__device__ void pass1_chunk(const FusedArgs& A, Smem<K, TM, R, NW, DR, NM>& S, int ch, const PairPos pp, R* __restrict__ wsc) {
  constexpr int KT = K / 16;
  const int lane = threadIdx.x & 63, g = lane >> 4, c = lane & 15;
  // chunk-wide values, in scalar registers
  const int start = __builtin_amdgcn_readfirstlane(S.ch_start[ch]);
  const int count = __builtin_amdgcn_readfirstlane(S.ch_count[ch]);

  double dxd, dyd, dzd;
  int atom;
  pair_delta(A, S, ch, pp, &dxd, &dyd, &dzd, &atom);
  const R dx = R(dxd), dy = R(dyd), dz = R(dzd);
  const R r = vsqrt(dx * dx + dy * dy + dz * dz);
  const R ir = vrcp(r);
  const R ux = dx * ir, uy = dy * ir, uz = dz * ir;
  R fc, dfc_unused;
  cutoff(r, R(A.pi_rc), &fc, &dfc_unused);
  if (atom < 0) fc = R(0);

  R h[8][4], dh[8][4];
  const R* __restrict__ layer =
      encoder_hidden<K, TM, R, NW, DR, NM, kWs>(A, S, S.ch_s[ch], r, chunk_table(A, S, ch), h, dh);
  v4<R> mo[KT], dmo[KT];
  encoder_out_rows<K, R, kWs>(layer, h, dh, mo, dmo);

  // moment: P[mm][col] += sum_pairs fc * a_mm(u) * m[pair][col], one MFMA
  // product per centre atom present in the chunk and 16-row tile of the
  // angular features (pairs of other atoms are masked to zero in the A
  // operand).  The features themselves are an MFMA product over the
  // monomials, F[pair][mm] = sum_m fc m_m(u_pair) Q[mm][m], whose result
  // registers (register q: pair drow(q, g), row c) are exactly the A operand
  // of the moment product; each lane forms only its own pair's monomials.
  constexpr int NA = DR / 16;
  static_assert(NM % 4 == 0, "monomial count must be a multiple of the MFMA k-step");
  v4<R> av[NA];
  int aa[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) aa[q] = __shfl(atom, drow<R>(q, g), 64);
  {
    R mono[NM];
    monomials_n<NM, false>(ux, uy, uz, mono, mono, mono, mono);
#pragma unroll
    for (int ta = 0; ta < NA; ++ta) av[ta] = v4<R>{0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < NM / 4; ++i) {
      // A[pair c][m = 4i + g] = fc m_m(u_c); B[m = 4i + g][row c] = Q[row][m]
      const R x = fc * pick4(g, mono[4 * i], mono[4 * i + 1], mono[4 * i + 2], mono[4 * i + 3]);
#pragma unroll
      for (int ta = 0; ta < NA; ++ta) av[ta] = mfma(x, S.qc[16 * ta + c][4 * i + g], av[ta]);
    }
  }
  const int a_first = __builtin_amdgcn_readfirstlane(S.pair_a[start]);
  const int a_last = __builtin_amdgcn_readfirstlane(S.pair_a[start + count - 1]);
  for (int a = a_first; a <= a_last; ++a) {
#pragma unroll
    for (int ta = 0; ta < NA; ++ta) {
      v4<R> pacc[KT];
#pragma unroll
      for (int Tc = 0; Tc < KT; ++Tc) pacc[Tc] = v4<R>{0, 0, 0, 0};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const R av_a = aa[q] == a ? av[ta][q] : R(0);
#pragma unroll
        for (int Tc = 0; Tc < KT; ++Tc) pacc[Tc] = mfma(av_a, mo[Tc][q], pacc[Tc]);
      }
      constexpr int DRS = moment_rows(DR, NM);
#pragma unroll
      for (int Tc = 0; Tc < KT; ++Tc)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int row = 16 * ta + drow<R>(q, g);
          if (16 * ta + 16 <= DRS || row < DRS) atomicAdd(&S.P[a][row][16 * Tc + c], pacc[Tc][q]);
        }
    }
  }

  if (kWs) {
    // workspace in the B-operand order pass 2 loads, contiguous per lane:
    // lane 16 g' + c' holds m[pair c'][16Tc + drow(i, g')] at 4 KT lane' +
    // 4 Tc + i (then the same for dm)
#pragma unroll
    for (int Tc = 0; Tc < KT; ++Tc)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int off = (16 * gof<R>(c) + drow<R>(q, g)) * (4 * KT) + Tc * 4 + qof<R>(c);
        wsc[off] = mo[Tc][q];
        wsc[K * 16 + off] = dmo[Tc][q];
      }
  }
}

// Inputs of pass 2 for one chunk: the workspace tiles (m, dm) in B-operand
// order and the neighbour position; loaded one chunk ahead.
template <int K, typename R>
struct Pass2In {
  R mB[K / 16][4], dmB[K / 16][4];
  PairPos pp;
};

template <int K, int TM, typename R, int NW, int DR, int NM>
__device__ __forceinline__ void pass2_load(const FusedArgs& A, const Smem<K, TM, R, NW, DR, NM>& S, int ch,
                                           const R* __restrict__ wsc, Pass2In<K, R>& in) {
  constexpr int VW = 16 / int(sizeof(R));
  constexpr int NV = K / 4 / VW;  // 16-byte loads per lane for m (and for dm)
  typedef R vw_t __attribute__((ext_vector_type(VW)));
  const int lane = threadIdx.x & 63;
  const vw_t* __restrict__ pm = reinterpret_cast<const vw_t*>(wsc + lane * (K / 4));
  const vw_t* __restrict__ pd = reinterpret_cast<const vw_t*>(wsc + K * 16 + lane * (K / 4));
  vw_t vm[NV], vd[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    vm[v] = pm[v];
    vd[v] = pd[v];
  }
#pragma unroll
  for (int Tc = 0; Tc < K / 16; ++Tc)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      in.mB[Tc][i] = vm[(Tc * 4 + i) / VW][(Tc * 4 + i) % VW];
      in.dmB[Tc][i] = vd[(Tc * 4 + i) / VW][(Tc * 4 + i) % VW];
    }
  in.pp = load_pair_pos(A, S, ch);
}

// Inputs of pass 2 for one chunk by recomputing the encoder instead of
// reading the workspace (the paper's mega-fusion, Section 3.4).
template <int K, int TM, typename R, int NW, int DR, int NM>
__device__ __forceinline__ void pass2_recompute(const FusedArgs& A, const Smem<K, TM, R, NW, DR, NM>& S, int ch,
                                                const PairPos& pp, Pass2In<K, R>& in) {
  double dxd, dyd, dzd;
  int atom;
  pair_delta(A, S, ch, pp, &dxd, &dyd, &dzd, &atom);
  const R dx = R(dxd), dy = R(dyd), dz = R(dzd);
  const R r = vsqrt(dx * dx + dy * dy + dz * dz);
  R h[8][4], dh[8][4];
  const R* __restrict__ layer = encoder_hidden(A, S, S.ch_s[ch], r, chunk_table(A, S, ch), h, dh);
  encoder_out_cols<K, R>(layer, h, dh, in.mB, in.dmB);
  in.pp = pp;
}

// F_j -= f_ij through the tile's table in LDS (open addressing by a
// multiplicative hash of j, linear probing); when every probe position of j
// is taken by other neighbours the contribution goes straight to HBM.
template <int K, int TM, typename R, int NW, int DR, int NM>
__device__ __forceinline__ void scatter_fj_tile(const FusedArgs& A, Smem<K, TM, R, NW, DR, NM>& S, int j, double fx,
                                                double fy, double fz) {
  constexpr int kProbes = 32;
  int slot = int((unsigned(j) * 0x9E3779B1u) >> 22);  // 10 bits: kFjSlots = 1024
  for (int p = 0; p < kProbes; ++p) {
    const int prev = atomicCAS(&S.u.fj.key[slot], -1, j);
    if (prev == -1 || prev == j) {
      atomicAdd(&S.u.fj.val[slot][0], -fx);
      atomicAdd(&S.u.fj.val[slot][1], -fy);
      atomicAdd(&S.u.fj.val[slot][2], -fz);
      return;
    }
    slot = (slot + 1) & (kFjSlots - 1);
  }
  atomicAdd(&A.forces[3 * (long long)j], -fx);
  atomicAdd(&A.forces[3 * (long long)j + 1], -fy);
  atomicAdd(&A.forces[3 * (long long)j + 2], -fz);
}

// Pass 2 on one chunk: W contractions, partial forces and scatter (F_j by
// global atomics, or with kTileFj through the tile's table).
template <int K, int TM, typename R, int NW, int DR, int NM, bool kTileFj = false>
__device__ void pass2_chunk(const FusedArgs& A, Smem<K, TM, R, NW, DR, NM>& S, int ch, const Pass2In<K, R>& in) {
  constexpr int KT = K / 16;
  const int lane = threadIdx.x & 63, g = lane >> 4, c = lane & 15;
  // chunk-wide values, in scalar registers
  const int start = __builtin_amdgcn_readfirstlane(S.ch_start[ch]);
  const int count = __builtin_amdgcn_readfirstlane(S.ch_count[ch]);

  const bool valid = c < count;
  int atom = -1, j = 0;
  double dx = 1.0, dy = 0.0, dz = 0.0;  // minimum image in float64, kept for the virial
  if (valid) {
    const int e = start + c;
    j = S.pair_j[e];
    atom = S.pair_a[e];
    dx = fold(in.pp.x - S.tpos[atom][0], A.box[0], A.inv_box[0]);
    dy = fold(in.pp.y - S.tpos[atom][1], A.box[1], A.inv_box[1]);
    dz = fold(in.pp.z - S.tpos[atom][2], A.box[2], A.inv_box[2]);
  }
  const R rx = R(dx), ry = R(dy), rz = R(dz);
  const R r = vsqrt(rx * rx + ry * ry + rz * rz);
  const R ir = vrcp(r);
  const R ux = rx * ir, uy = ry * ir, uz = rz * ir;
  R fc, dfc;
  cutoff(r, R(A.pi_rc), &fc, &dfc);
  if (!valid) fc = dfc = R(0);

  // (W m) and (W dm) for this column's own centre atom, one 16-row tile of
  // the angular features at a time
  constexpr int NA = DR / 16;
  v4<R> wm[NA], wdm[NA];
#pragma unroll
  for (int ta = 0; ta < NA; ++ta) wm[ta] = wdm[ta] = v4<R>{0, 0, 0, 0};
  const int a_first = __builtin_amdgcn_readfirstlane(S.pair_a[start]);
  const int a_last = __builtin_amdgcn_readfirstlane(S.pair_a[start + count - 1]);
  for (int a = a_first; a <= a_last; ++a) {
#pragma unroll
    for (int ta = 0; ta < NA; ++ta) {
      v4<R> t1 = v4<R>{0, 0, 0, 0}, t2 = v4<R>{0, 0, 0, 0};
#pragma unroll
      for (int Tc = 0; Tc < KT; ++Tc)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          constexpr int DRS = moment_rows(DR, NM);
          const R w = 16 * ta + 16 <= DRS || 16 * ta + c < DRS ? S.P[a][16 * ta + c][16 * Tc + drow<R>(i, g)] : R(0);
          t1 = mfma(w, in.mB[Tc][i], t1);
          t2 = mfma(w, in.dmB[Tc][i], t2);
        }
      if (atom == a) {
        wm[ta] = t1;
        wdm[ta] = t2;
      }
    }
  }

  // angular features a_mm and gradients for rows mm = 16 ta + drow(q, g) of
  // this pair, accumulated monomial by monomial so that each monomial and
  // its gradient are live only for their own step
  R mono[NM], gx[NM], gy[NM], gz[NM];
  monomials_n<NM, true>(ux, uy, uz, mono, gx, gy, gz);
  R fv[NA][4], fgx[NA][4], fgy[NA][4], fgz[NA][4];
#pragma unroll
  for (int ta = 0; ta < NA; ++ta)
#pragma unroll
    for (int q = 0; q < 4; ++q) fv[ta][q] = fgx[ta][q] = fgy[ta][q] = fgz[ta][q] = R(0);
#pragma unroll
  for (int m = 0; m < NM; ++m)
#pragma unroll
    for (int ta = 0; ta < NA; ++ta)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const R co = S.qc[16 * ta + drow<R>(q, g)][m];
        fv[ta][q] += co * mono[m];
        fgx[ta][q] += co * gx[m];
        fgy[ta][q] += co * gy[m];
        fgz[ta][q] += co * gz[m];
      }
  R s = 0, tx = 0, ty = 0, tz = 0;
#pragma unroll
  for (int ta = 0; ta < NA; ++ta)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const R v = fc * wm[ta][q];                       // v = W g
      const R wg = dfc * wm[ta][q] + fc * wdm[ta][q];   // W g'
      s += fv[ta][q] * wg;
      tx += fgx[ta][q] * v;
      ty += fgy[ta][q] * v;
      tz += fgz[ta][q] * v;
    }
#pragma unroll
  for (int o = 16; o <= 32; o <<= 1) {
    s += __shfl_xor(s, o, 64);
    tx += __shfl_xor(tx, o, 64);
    ty += __shfl_xor(ty, o, 64);
    tz += __shfl_xor(tz, o, 64);
  }
  // f = s u + (I - u u^T) t / r  (Eq. 10, reassociated), accumulated in float64
  const R ut = ux * tx + uy * ty + uz * tz;
  const double fx = double(s * ux + (tx - ut * ux) * ir);
  const double fy = double(s * uy + (ty - ut * uy) * ir);
  const double fz = double(s * uz + (tz - ut * uz) * ir);
  if (valid) {
    if (g == 0) {
      if constexpr (kTileFj) {
        scatter_fj_tile(A, S, j, fx, fy, fz);
      } else {
        atomicAdd(&A.forces[3 * (long long)j], -fx);
        atomicAdd(&A.forces[3 * (long long)j + 1], -fy);
        atomicAdd(&A.forces[3 * (long long)j + 2], -fz);
      }
    } else if (g == 1) {
      atomicAdd(&S.Fi[atom][0], fx);
      atomicAdd(&S.Fi[atom][1], fy);
      atomicAdd(&S.Fi[atom][2], fz);
    } else if (g == 2) {
      atomicAdd(&S.Wi[atom][0], -dx * fx);
      atomicAdd(&S.Wi[atom][1], -dx * fy);
      atomicAdd(&S.Wi[atom][2], -dx * fz);
      atomicAdd(&S.Wi[atom][3], -dy * fx);
      atomicAdd(&S.Wi[atom][4], -dy * fy);
    } else {
      atomicAdd(&S.Wi[atom][5], -dy * fz);
      atomicAdd(&S.Wi[atom][6], -dz * fx);
      atomicAdd(&S.Wi[atom][7], -dz * fy);
      atomicAdd(&S.Wi[atom][8], -dz * fz);
    }
  }
}

// Radial kernel of the unfused configuration (Eq. 2 as a kernel of its own)
// on one chunk: g = fc(r) MLP(r) and dg/dr of each pair from the distance
// the setup kernel stored for its neighbour-list entry, written back by
// entry.  The chunk's pair slots hold entry indices relative to the tile's
// first entry.
template <int K, int TM, typename R, int NW, int DR, int NM>
__device__ void radial_chunk(const FusedArgs& A, const Smem<K, TM, R, NW, DR, NM>& S, int ch) {
  constexpr int KT = K / 16;
  const int lane = threadIdx.x & 63, g = lane >> 4, c = lane & 15;
  const bool valid = c < S.ch_count[ch];
  const long long e = S.row_beg[0] + (valid ? S.pair_j[S.ch_start[ch] + c] : 0);
  const R r = valid ? R(A.geo[4 * e + 3]) : R(1);
  R fc, dfc;
  cutoff(r, R(A.pi_rc), &fc, &dfc);
  if (!valid) fc = dfc = R(0);
  R h[8][4], dh[8][4];
  const R* __restrict__ layer = encoder_hidden(A, S, S.ch_s[ch], r, chunk_table(A, S, ch), h, dh);
  R mB[KT][4], dmB[KT][4];
  encoder_out_cols<K, R>(layer, h, dh, mB, dmB);
  if (valid) {
    R* __restrict__ gr = static_cast<R*>(A.grad) + e * K;
    R* __restrict__ gp = static_cast<R*>(A.gprime) + e * K;
#pragma unroll
    for (int Tc = 0; Tc < KT; ++Tc)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int col = 16 * Tc + drow<R>(q, g);
        gr[col] = fc * mB[Tc][q];
        gp[col] = dfc * mB[Tc][q] + fc * dmB[Tc][q];
      }
  }
}

// Descriptor value x[in] = vec(G)[in] of tile atom a (Eq. 5): the l = 0
// block is linear, a block l >= 1 (angular rows lrow[l] .. lrow[l+1]-1) is
// the quadratic form sum_m rw[m] P[m][col]^2 with the block's diagonal
// metric (1 for the irreducible basis, the multinomial coefficients for the
// Cartesian one).
template <int K, int TM, typename R, int NW, int DR, int NM>
__device__ __forceinline__ R descriptor_value(const FusedArgs& A, const Smem<K, TM, R, NW, DR, NM>& S, int a, int in) {
  const int l = in / K, col = in % K;
  if (l == 0) return S.P[a][0][col];
  R v = 0;
  for (int mm = A.lrow[l]; mm < A.lrow[l + 1]; ++mm) v += S.rw[mm] * S.P[a][mm][col] * S.P[a][mm][col];
  return v;
}

// W = dE/dP (Eq. 7) for tile atom a from dE/dx[in]: W[0][col] = dE/dG[0][col],
// W[m][col] = 2 dE/dG[l][col] rw[m] P[m][col]; overwrites P.
template <int K, int TM, typename R, int NW, int DR, int NM>
__device__ __forceinline__ void adjoint_from_grad(const FusedArgs& A, Smem<K, TM, R, NW, DR, NM>& S, int a, int in,
                                                  R d) {
  const int l = in / K, col = in % K;
  if (l == 0) {
    S.P[a][0][col] = d;
  } else {
    for (int mm = A.lrow[l]; mm < A.lrow[l + 1]; ++mm) S.P[a][mm][col] *= R(2) * S.rw[mm] * d;
  }
}

// Weight fragments of the head products, consumed in groups of 16 k-steps.
// Group G of a wavefront that owns output rows (w < 4): the first layer's
// k-steps 16G .. 16G+15, then the hidden layers forward, the hidden layers
// backward (A_t^T), then the A0^T output tiles tt = w, w + NW, ...; the
// other wavefronts only take A0^T tiles.  Element ks of a group is at
// p[ks * stride * 64]; n is the group's k-step count (0 past the end).
template <typename R>
struct HeadGroup {
  const R* p;
  int stride, n;
};

template <typename R>
__device__ __forceinline__ HeadGroup<R> head_group(int G, bool rw, int w, int nw, int nin, int nhid,
                                                   const R* __restrict__ A0f, const R* __restrict__ A0Tf,
                                                   const R* __restrict__ hid) {
  constexpr int RW = kHeadWidth;
  constexpr int HS = 2 * RW * RW + RW;
  const int lane = threadIdx.x & 63;
  const int tin = nin / 16, k0 = nin / 4, nl0 = (k0 + 15) / 16;
  if (rw) {
    if (G < nl0) return {A0f + (64 * G + w) * 64 + lane, 4, k0 - 16 * G < 16 ? k0 - 16 * G : 16};
    G -= nl0;
    if (G < nhid) return {hid + G * HS + w * 64 + lane, 4, 16};
    G -= nhid;
    if (G < nhid) return {hid + (nhid - 1 - G) * HS + RW * RW + w * 64 + lane, 4, 16};
    G -= nhid;
  }
  const int tt = w + nw * G;
  if (tt < tin) return {A0Tf + tt * 64 + lane, tin, 16};
  return {A0Tf, 0, 0};
}

template <typename R>
__device__ __forceinline__ void head_load(const HeadGroup<R>& d, R (&f)[16]) {
#pragma unroll
  for (int ks = 0; ks < 16; ++ks) f[ks] = ks < d.n ? d.p[ks * d.stride * 64] : R(0);
}

// Descriptor (Eq. 5), head forward and backward (Eq. 6) and W = dE/dP
// (Eq. 7) for the tile on MFMA: the tile's atoms are the 16 columns of every
// product and wavefront w < 4 owns rows 16w..16w+15 of each 64-wide layer.
// Activations live in LDS feature-major ([feature][atom]) so that B-operand
// reads are contiguous; pre-activations stay in registers for the backward
// pass.  Each wavefront streams its weight fragments one 16-k-step group
// ahead of the products (the first group before the descriptor is formed),
// so a layer's fragments arrive while the previous layer and its barriers
// run.  With kRegress (the regression kernel of the three-kernel and unfused
// configurations) the descriptor comes from HBM and dE/dx goes back to HBM
// in its place instead of forming W.
template <int K, int TM, typename R, int NW, int DR, int NM, bool kRegress>
__device__ void head_stage(const FusedArgs& A, Smem<K, TM, R, NW, DR, NM>& S) {
  constexpr int RW = kHeadWidth;
  constexpr int HS = 2 * RW * RW + RW;  // one hidden layer: A_t and A_t^T fragments, c_t
  constexpr int NC = TM > 16 ? 32 : 16;  // atom columns: one or two groups of 16
  constexpr int CG = NC / 16;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 4, c = lane & 15, w = tid >> 6;
  const int na = S.na;
  const int nin = (A.lmax + 1) * K;
  const int tin = nin / 16;
  const int nhid = A.reg_hidden - 1;
  const int rho = A.reg_cond ? S.tile_species : 0;
  const R* __restrict__ A0f = static_cast<const R*>(A.head) + (long long)rho * A.head_stride;  // A0 fragments
  const R* __restrict__ A0Tf = A0f + RW * nin;                                               // A0^T fragments
  const R* __restrict__ c0 = A0Tf + RW * nin;
  const R* __restrict__ hid = c0 + RW;
  const R* __restrict__ aout = hid + nhid * HS;
  // this lane's result rows are 16 w + drow(q, g); with more than 4
  // wavefronts the others only join the barriers of the row-parallel steps
  // and take A0^T tiles.  Each weight fragment multiplies the CG column
  // groups of atoms.
  const bool rw = w < RW / 16;
  int G = 0;
  R fcur[16], fnext[16];
  head_load(head_group(G, rw, w, NW, nin, nhid, A0f, A0Tf, hid), fnext);
  // next group: the fetched one becomes current and the one after it is fetched
#define ADVANCE()                                                          \
  do {                                                                     \
    _Pragma("unroll") for (int ks_ = 0; ks_ < 16; ++ks_) fcur[ks_] = fnext[ks_]; \
    ++G;                                                                   \
    head_load(head_group(G, rw, w, NW, nin, nhid, A0f, A0Tf, hid), fnext); \
  } while (0)

  // B-operand reads from the feature-major activations: element
  // [16 (k >> 2) + drow(k & 3, g)][16 cg + c] sits at a per-lane base plus an
  // offset that depends on k and cg only, so every read is that base with an
  // immediate offset instead of an address register of its own (no
  // __restrict__: yT and gT are also written through S between the barriers)
  const R* xl = &S.u.hd.xT[0][0] + drow<R>(0, g) * NC + c;
  const R* yl = &S.u.hd.yT[0][0] + drow<R>(0, g) * NC + c;
  const R* gl = &S.u.hd.gT[0][0] + drow<R>(0, g) * NC + c;
#define BOFF(k) ((16 * ((k) >> 2) + drow<R>((k) & 3, 0)) * NC)

  R* __restrict__ gbuf = kRegress ? static_cast<R*>(A.gbuf) + (long long)S.a0 * nin : nullptr;
  for (int u = tid; u < NC * nin; u += (64 * NW)) {
    const int a = u % NC, in = u / NC;
    R v = 0;
    if (a < na) v = kRegress ? gbuf[(long long)a * nin + in] : descriptor_value(A, S, a, in);
    S.u.hd.xT[in][a] = v;
  }
  __syncthreads();

#define ROW(q) (16 * w + drow<R>(q, g))

  // layer 0: z0 = A0 x + c0, over nin / 4 k-steps in groups of 16 with two
  // accumulators alternating
  v4<R> z0[CG];
#pragma unroll
  for (int cg = 0; cg < CG; ++cg) z0[cg] = v4<R>{0, 0, 0, 0};
  if (rw) {
    v4<R> z0b[CG];
#pragma unroll
    for (int cg = 0; cg < CG; ++cg) {
      z0[cg] = v4<R>{c0[ROW(0)], c0[ROW(1)], c0[ROW(2)], c0[ROW(3)]};
      z0b[cg] = v4<R>{0, 0, 0, 0};
    }
    const int k0 = nin / 4;
    for (int kb = 0; kb < k0; kb += 16) {
      ADVANCE();
      const R* xk = xl + 4 * kb * NC;  // kb is a multiple of 16
#pragma unroll
      for (int ks = 0; ks < 16; ks += 2) {
        if (kb + ks < k0) {
#pragma unroll
          for (int cg = 0; cg < CG; ++cg) {
            z0[cg] = mfma(fcur[ks], xk[BOFF(ks) + 16 * cg], z0[cg]);
            z0b[cg] = mfma(fcur[ks + 1], xk[BOFF(ks + 1) + 16 * cg], z0b[cg]);
          }
        }
      }
    }
#pragma unroll
    for (int cg = 0; cg < CG; ++cg) {
      z0[cg] += z0b[cg];
#pragma unroll
      for (int q = 0; q < 4; ++q) S.u.hd.yT[ROW(q)][16 * cg + c] = z0[cg][q] * sigmoid(z0[cg][q]);
    }
  }
  __syncthreads();

  // residual layers: y <- y + silu(A_t y + c_t)
  v4<R> zeta[kMaxHidden][CG];
#pragma unroll
  for (int t = 1; t < kMaxHidden; ++t) {
    if (t >= A.reg_hidden) break;
    const R* __restrict__ ct = hid + (t - 1) * HS + 2 * RW * RW;
    v4<R> z[CG];
#pragma unroll
    for (int cg = 0; cg < CG; ++cg) z[cg] = v4<R>{0, 0, 0, 0};
    if (rw) {
      ADVANCE();
#pragma unroll
      for (int cg = 0; cg < CG; ++cg) z[cg] = v4<R>{ct[ROW(0)], ct[ROW(1)], ct[ROW(2)], ct[ROW(3)]};
#pragma unroll
      for (int ks = 0; ks < 16; ++ks)
#pragma unroll
        for (int cg = 0; cg < CG; ++cg)
          z[cg] = mfma(fcur[ks], yl[BOFF(ks) + 16 * cg], z[cg]);
    }
#pragma unroll
    for (int cg = 0; cg < CG; ++cg) zeta[t][cg] = z[cg];
    __syncthreads();
    if (rw) {
#pragma unroll
      for (int cg = 0; cg < CG; ++cg)
#pragma unroll
        for (int q = 0; q < 4; ++q) S.u.hd.yT[ROW(q)][16 * cg + c] += z[cg][q] * sigmoid(z[cg][q]);
    }
    __syncthreads();
  }
  if (tid < na) {
    R e = aout[RW];
    for (int o = 0; o < RW; ++o) e += aout[o] * S.u.hd.yT[o][tid];
    S.Ei[tid] = double(e);
  }

  // backward: d <- d + A_t^T (silu'(zeta_t) d), starting from d = a_out
  v4<R> d[CG];
#pragma unroll
  for (int cg = 0; cg < CG; ++cg)
    d[cg] = rw ? v4<R>{aout[ROW(0)], aout[ROW(1)], aout[ROW(2)], aout[ROW(3)]} : v4<R>{0, 0, 0, 0};
#pragma unroll
  for (int t = kMaxHidden - 1; t >= 1; --t) {
    if (t >= A.reg_hidden) continue;
    if (rw) {
#pragma unroll
      for (int cg = 0; cg < CG; ++cg)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const R z = zeta[t][cg][q], sg = sigmoid(z);
          S.u.hd.gT[ROW(q)][16 * cg + c] = silu_slope(z, sg) * d[cg][q];
        }
    }
    __syncthreads();
    if (rw) {
      ADVANCE();
      v4<R> acc[CG];
#pragma unroll
      for (int cg = 0; cg < CG; ++cg) acc[cg] = v4<R>{0, 0, 0, 0};
#pragma unroll
      for (int ks = 0; ks < 16; ++ks)
#pragma unroll
        for (int cg = 0; cg < CG; ++cg)
          acc[cg] = mfma(fcur[ks], gl[BOFF(ks) + 16 * cg], acc[cg]);
#pragma unroll
      for (int cg = 0; cg < CG; ++cg) d[cg] += acc[cg];
    }
    __syncthreads();
  }
  if (rw) {
#pragma unroll
    for (int cg = 0; cg < CG; ++cg)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const R z = z0[cg][q], sg = sigmoid(z);
        S.u.hd.gT[ROW(q)][16 * cg + c] = silu_slope(z, sg) * d[cg][q];
      }
  }
  __syncthreads();
  // dE/dx = A0^T g0, then W[0][col] = dE/dG[0][col], W[m][col] = 2 dE/dG[l][col] P[m][col]
  for (int tt = w; tt < tin; tt += NW) {
    ADVANCE();
    v4<R> acc[CG];
#pragma unroll
    for (int cg = 0; cg < CG; ++cg) acc[cg] = v4<R>{0, 0, 0, 0};
#pragma unroll
    for (int ks = 0; ks < 16; ++ks) {
#pragma unroll
      for (int cg = 0; cg < CG; ++cg)
        acc[cg] = mfma(fcur[ks], gl[BOFF(ks) + 16 * cg], acc[cg]);
    }
#pragma unroll
    for (int cg = 0; cg < CG; ++cg) {
      const int a = 16 * cg + c;
      if (a < na) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int in = 16 * tt + drow<R>(q, g);
          if (kRegress)
            gbuf[(long long)a * nin + in] = acc[cg][q];
          else
            adjoint_from_grad(A, S, a, in, acc[cg][q]);
        }
      }
    }
  }
  __syncthreads();
#undef BOFF
#undef ROW
#undef ADVANCE
}

// First-layer weights (w0, b0) of the tile's encoder tables, one per
// neighbour species, into LDS.
template <int K, int TM, typename R, int NW, int DR, int NM>
__device__ __forceinline__ void stage_first_layer(const FusedArgs& A, Smem<K, TM, R, NW, DR, NM>& S,
                                                  const R* __restrict__ enc) {
  for (int u = threadIdx.x; u < A.C * 2 * kEncWidth; u += 64 * NW) {
    const int sj = u / (2 * kEncWidth), rem = u % (2 * kEncWidth);
    const int si = S.tile_species;
    const int tau = A.enc_cond == 2 ? si * A.C + sj : (A.enc_cond == 1 ? sj : 0);
    S.u.l0[sj][rem / kEncWidth][rem % kEncWidth] = enc[(long long)tau * A.enc_stride + rem];
  }
}

// What one launch does (Section 3.4 fusion configurations): the single
// kernel that caches (m, dm) between its two passes or recomputes them in
// pass 2; one of the three kernels of the partial configuration: encoding
// (Eqs. 1-5, G to HBM), regression (Eq. 6, E and dE/dG to HBM) and
// derivation (Eqs. 7-10, recomputing P); or the radial kernel of the unfused
// configuration (Eq. 2 alone, which uses the regression kernel as well).
enum Mode { kCached = 0, kRecompute = 1, kEncode = 2, kRegress = 3, kDerive = 4, kRadial = 5, kCachedTileFj = 6 };
static_assert(kCachedTileFj == kModeCachedTileFj, "mode number of the tile-reduced scatter");
static_assert(kRegress == kModeRegress && kRadial == kModeRadial, "mode numbers of the unfused configuration");

template <int K, int TM, typename R, int NW, int DR, int NM, int MODE>
__global__ __launch_bounds__(64 * NW, 1) void k_fused(FusedArgs A) {
  static_assert(TM <= 64, "the bucket table gives one lane to each atom of a tile");
  extern __shared__ __align__(16) unsigned char smem_raw[];
  Smem<K, TM, R, NW, DR, NM>& S = *reinterpret_cast<Smem<K, TM, R, NW, DR, NM>*>(smem_raw);
  const int tid = threadIdx.x, wave = tid >> 6;
  const long long chunk_elems = 2LL * K * 16;
  R* __restrict__ ws_slot = static_cast<R*>(A.ws) + (long long)blockIdx.x * A.ws_slot;
  const R* __restrict__ enc = static_cast<const R*>(A.enc);
  const R* __restrict__ qc = static_cast<const R*>(A.qc);

  for (int u = tid; u < DR * NM; u += (64 * NW)) S.qc[u / NM][u % NM] = qc[u];
  for (int u = tid; u < DR; u += 64 * NW) S.rw[u] = qc[DR * NM + u];

  // XCD-aware assignment: blocks are dispatched round-robin over the 8 XCDs,
  // so block b works on the b%8-th contiguous eighth of the tile list and
  // spatially adjacent tiles share an L2.
  const int G = gridDim.x;
  const int nx = (G % 8 == 0) ? 8 : 1;
  const int xcd = blockIdx.x % nx, slot = blockIdx.x / nx, per = G / nx;
  const int lo = int((long long)A.n_tiles * xcd / nx), hi = int((long long)A.n_tiles * (xcd + 1) / nx);

  for (int tile = lo + slot; tile < hi; tile += per) {
    // ---- A: stage atoms and rows -----------------------------------------
    // The rows of consecutive sorted atoms are one contiguous run of the
    // neighbour list, and each row is grouped by neighbour species, so the
    // bucket position of an entry follows from a block-wide prefix count of
    // active entries; every thread handles 8 consecutive entries.
    if (tid == 0) {
      int s = 0;
      while (s + 1 < A.C && tile >= A.tile_start[s + 1]) ++s;
      const int first = A.species_start[s] + (tile - A.tile_start[s]) * A.tile_atoms;
      const int rem = A.species_start[s + 1] - first;
      S.tile_species = s;
      S.na = rem < A.tile_atoms ? rem : A.tile_atoms;
      S.a0 = first;
    }
    __syncthreads();
    const int na = S.na;
    const int a0 = S.a0;
    if (tid < TM) {
      if (tid < na) {
        const int o = A.perm[a0 + tid];
        S.orig[tid] = o;
        if (A.list.idx16) centre_cells(A.list, A.list.key[o], S.cand[tid]);
        S.tpos[tid][0] = A.pos[3 * (long long)o];
        S.tpos[tid][1] = A.pos[3 * (long long)o + 1];
        S.tpos[tid][2] = A.pos[3 * (long long)o + 2];
      }
#pragma unroll
      for (int k = 0; k < 3; ++k) S.Fi[tid][k] = 0.0;
#pragma unroll
      for (int k = 0; k < 9; ++k) S.Wi[tid][k] = 0.0;
      S.Ei[tid] = 0.0;
    }
    int nch = 0;
    if constexpr (MODE != kRegress) {
    stage_first_layer(A, S, enc);
    if (tid <= TM) {
      const int k = tid < na ? tid : na;
      S.ent_base[tid] = int(A.offsets[a0 + k] - A.offsets[a0]);
      if (tid == 0) S.row_beg[0] = A.offsets[a0];
    }
    for (int u = tid; u < kMaxSpecies * TM; u += (64 * NW)) S.cnt[u / TM][u % TM] = 0;
    if constexpr (MODE != kRadial)
      for (int u = tid; u < TM * moment_rows(DR, NM) * (K + 1); u += (64 * NW)) (&S.P[0][0][0])[u] = R(0);
    __syncthreads();
    const int nent = S.ent_base[na];
    const long long ebase = S.row_beg[0];
    constexpr int kPer = tile_entry_cap(TM) / (64 * NW);
    static_assert(kPer * 64 * NW == tile_entry_cap(TM), "every listed entry of a tile needs a thread");
    int ej[kPer], ea[kPer], es[kPer];
    int my_active = 0;
    {
      const int e0 = tid * kPer;
      int a = 0;
      while (a + 1 < na && e0 >= S.ent_base[a + 1]) ++a;
#pragma unroll
      for (int k = 0; k < kPer; ++k) {
        while (a + 1 < na && e0 + k >= S.ent_base[a + 1]) ++a;
        ea[k] = a;
      }
      if (A.list.idx32) {
#pragma unroll
        for (int k = 0; k < kPer; ++k) ej[k] = e0 + k < nent ? A.list.idx32[ebase + e0 + k] : -1;
      } else {
        // coded entries: bucket start through the centre's candidate cells,
        // then the permutation (each level's loads issued together)
        unsigned code[kPer];
        int slot[kPer];
#pragma unroll
        for (int k = 0; k < kPer; ++k) code[k] = e0 + k < nent ? A.list.idx16[ebase + e0 + k] : 0u;
#pragma unroll
        for (int k = 0; k < kPer; ++k) slot[k] = e0 + k < nent ? code_slot(A.list, S.cand[ea[k]], code[k]) : -1;
#pragma unroll
        for (int k = 0; k < kPer; ++k) ej[k] = slot[k] >= 0 ? A.list.perm[slot[k]] : -1;
      }
#pragma unroll
      for (int k = 0; k < kPer; ++k) {
        const int e = e0 + k;
        a = ea[k];
        es[k] = -1;
        const int j = ej[k];
        if (j >= 0) {
          bool active;
          if constexpr (MODE == kRadial) {
            // the setup kernel marked entries beyond the cutoff
            active = A.geo[4 * (ebase + e) + 3] >= 0.0;
          } else {
            const double dx = fold(A.pos[3 * (long long)j] - S.tpos[a][0], A.box[0], A.inv_box[0]);
            const double dy = fold(A.pos[3 * (long long)j + 1] - S.tpos[a][1], A.box[1], A.inv_box[1]);
            const double dz = fold(A.pos[3 * (long long)j + 2] - S.tpos[a][2], A.box[2], A.inv_box[2]);
            active = dx * dx + dy * dy + dz * dz < A.rc2;
          }
          if (active) {
            es[k] = A.types[j];
            atomicAdd(&S.cnt[es[k]][a], 1);
            ++my_active;
          }
        }
      }
    }
    // exclusive prefix of active entries over the block (entry order)
    int prefix;
    {
      int inc = my_active;
      const int ln = tid & 63;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int t = __shfl_up(inc, o, 64);
        if (ln >= o) inc += t;
      }
      if (ln == 63) S.wsum[wave] = inc;
      __syncthreads();
      prefix = inc - my_active;
      for (int w = 0; w < wave; ++w) prefix += S.wsum[w];
    }
    if (wave == 0) {
      // Bucket layout (species-major, atoms in order), chunk table, and the
      // offset turning an entry's block-wide active prefix (atom-major) into
      // its bucket slot: base[s][a] = (active entries of buckets before
      // (s, a) in species-major order) - (active entries before (a, s) in
      // atom-major order).  Lane a holds atom a; one lane scan per species.
      const int ln = tid;
      int run = 0, nchunk = 0, cum = 0;  // cum: this atom's entries of the species so far
      for (int s = 0; s < A.C; ++s) {
        const int x = ln < na ? S.cnt[s][ln] : 0;
        int inc = x;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int t = __shfl_up(inc, o, 64);
          if (ln >= o) inc += t;
        }
        const int tot = __shfl(inc, 63, 64);
        if (ln < na) S.base[s][ln] = run + inc - x - cum;
        cum += x;
        const int nb = (tot + 15) >> 4;
        for (int k = ln; k < nb; k += 64) {
          S.ch_start[nchunk + k] = run + 16 * k;
          S.ch_count[nchunk + k] = (unsigned char)(tot - 16 * k < 16 ? tot - 16 * k : 16);
          S.ch_s[nchunk + k] = (unsigned char)s;
        }
        nchunk += nb;
        run += tot;
      }
      // cum is now this atom's row total; subtract the atom-major row start
      int inc = cum;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int t = __shfl_up(inc, o, 64);
        if (ln >= o) inc += t;
      }
      const int row_start = inc - cum;
      if (ln < na)
        for (int s = 0; s < A.C; ++s) S.base[s][ln] -= row_start;
      if (ln == 0) {
        S.n_chunks = nchunk;
        S.next_chunk[0] = NW;  // chunk w < NW starts on wavefront w
        S.next_chunk[1] = NW;
        S.n_active = run;
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      if (es[k] >= 0) {
        const int s = es[k], a = ea[k];
        const int p = S.base[s][a] + prefix;
        // the list builder groups every row by species, so p always lies in
        // the (species, atom) run; the bound only keeps LDS accesses in range
        if (p >= 0 && p < S.n_active) {
          S.pair_j[p] = MODE == kRadial ? tid * kPer + k : ej[k];
          S.pair_a[p] = (unsigned char)a;
        }
        ++prefix;
      }
    }
    __syncthreads();

    // ---- B: pass 1 ---------------------------------------------------------
    nch = S.n_chunks;
    if constexpr (MODE == kRadial) {
      int ch = wave;
      while (ch < nch) {
        const int ch2 = grab_chunk(&S.next_chunk[0]);
        radial_chunk<K, TM, R, NW, DR, NM>(A, S, ch);
        ch = ch2;
      }
      if (tid == 0) atomicAdd(&A.counters[0], (unsigned long long)S.n_active);
      __syncthreads();
      continue;
    } else {
      constexpr bool kWs = MODE == kCached || MODE == kCachedTileFj || MODE == kDerive;
      int ch = wave;
      PairPos next = ch < nch ? load_pair_pos(A, S, ch) : PairPos{0.0, 0.0, 0.0};
      while (ch < nch) {
        const PairPos cur = next;
        const int ch2 = grab_chunk(&S.next_chunk[0]);
        if (ch2 < nch) next = load_pair_pos(A, S, ch2);
        pass1_chunk<K, TM, R, NW, DR, NM, kWs>(A, S, ch, cur, ws_slot + ch * chunk_elems);
        ch = ch2;
      }
    }
    __syncthreads();
    }  // MODE != kRegress

    // ---- C: descriptor, head, W ------------------------------------------
    if constexpr (MODE == kCached || MODE == kCachedTileFj || MODE == kRecompute) {
      head_stage<K, TM, R, NW, DR, NM, false>(A, S);
    } else if constexpr (MODE == kRegress) {
      head_stage<K, TM, R, NW, DR, NM, true>(A, S);
    } else if constexpr (MODE == kEncode || MODE == kDerive) {
      // encoding kernel: G to HBM; derivation kernel: W from dE/dG in HBM
      const int nin = (A.lmax + 1) * K;
      R* __restrict__ gbuf = static_cast<R*>(A.gbuf) + (long long)a0 * nin;
      for (int u = tid; u < na * nin; u += 64 * NW) {
        const int a = u / nin, in = u % nin;
        if constexpr (MODE == kEncode)
          gbuf[u] = descriptor_value(A, S, a, in);
        else
          adjoint_from_grad(A, S, a, in, gbuf[u]);
      }
      __syncthreads();
    }

    // ---- D: pass 2 ---------------------------------------------------------
    if constexpr (MODE == kCached || MODE == kCachedTileFj || MODE == kDerive) {
      constexpr bool kTileFj = MODE == kCachedTileFj;
      if constexpr (kTileFj) {
        // the head is done with the union: an empty table for this tile
        for (int u = tid; u < kFjSlots; u += 64 * NW) {
          S.u.fj.key[u] = -1;
          S.u.fj.val[u][0] = S.u.fj.val[u][1] = S.u.fj.val[u][2] = 0.0;
        }
        __syncthreads();
      }
      // inputs of the next chunk are loaded while this one is processed
      int ch = wave;
      Pass2In<K, R> next;
      if (ch < nch) pass2_load(A, S, ch, ws_slot + ch * chunk_elems, next);
      while (ch < nch) {
        const Pass2In<K, R> cur = next;
        const int ch2 = grab_chunk(&S.next_chunk[1]);
        if (ch2 < nch) pass2_load(A, S, ch2, ws_slot + ch2 * chunk_elems, next);
        pass2_chunk<K, TM, R, NW, DR, NM, kTileFj>(A, S, ch, cur);
        ch = ch2;
      }
      if constexpr (kTileFj) {
        // one atomic per distinct neighbour of the tile instead of one per pair
        __syncthreads();
        for (int u = tid; u < kFjSlots; u += 64 * NW) {
          const int j = S.u.fj.key[u];
          if (j >= 0) {
            atomicAdd(&A.forces[3 * (long long)j], S.u.fj.val[u][0]);
            atomicAdd(&A.forces[3 * (long long)j + 1], S.u.fj.val[u][1]);
            atomicAdd(&A.forces[3 * (long long)j + 2], S.u.fj.val[u][2]);
          }
        }
      }
    } else if constexpr (MODE == kRecompute) {
      // the head's activations overwrote the first-layer weights in LDS
      stage_first_layer(A, S, enc);
      __syncthreads();
      int ch = wave;
      PairPos next = ch < nch ? load_pair_pos(A, S, ch) : PairPos{0.0, 0.0, 0.0};
      while (ch < nch) {
        const PairPos cur = next;
        const int ch2 = grab_chunk(&S.next_chunk[1]);
        if (ch2 < nch) next = load_pair_pos(A, S, ch2);
        Pass2In<K, R> in;
        pass2_recompute(A, S, ch, cur, in);
        pass2_chunk<K, TM, R, NW, DR, NM>(A, S, ch, in);
        ch = ch2;
      }
    }
    __syncthreads();

    // ---- E: outputs --------------------------------------------------------
    constexpr bool kEnergy = MODE == kCached || MODE == kCachedTileFj || MODE == kRecompute || MODE == kRegress;
    constexpr bool kForces = MODE == kCached || MODE == kCachedTileFj || MODE == kRecompute || MODE == kDerive;
    if (tid < na) {
      const long long o = S.orig[tid];
      if (kEnergy && A.energy) A.energy[o] = S.Ei[tid];
      if (kForces) {
        if (A.virial) {
#pragma unroll
          for (int k = 0; k < 9; ++k) A.virial[9 * o + k] = S.Wi[tid][k];
        }
        atomicAdd(&A.forces[3 * o], S.Fi[tid][0]);
        atomicAdd(&A.forces[3 * o + 1], S.Fi[tid][1]);
        atomicAdd(&A.forces[3 * o + 2], S.Fi[tid][2]);
      }
    }
    if (wave == 0 && MODE != kEncode) {
      double v[10];
      const bool own = tid < na;
      v[0] = kEnergy && own ? S.Ei[tid] : 0.0;
#pragma unroll
      for (int k = 0; k < 9; ++k) v[1 + k] = kForces && own ? S.Wi[tid][k] : 0.0;
#pragma unroll
      for (int k = 0; k < 10; ++k)
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) v[k] += __shfl_xor(v[k], o, 64);
      if (tid < 10) {
        double mine = v[0];
#pragma unroll
        for (int k = 1; k < 10; ++k)
          if (tid == k) mine = v[k];
        atomicAdd(&A.totals[tid], mine);
      }
      if (tid == 0 && kForces) atomicAdd(&A.counters[0], (unsigned long long)S.n_active);
    }
    __syncthreads();
  }
}

template <int K, int TM, typename R, int NW, int DR, int NM, int MODE>
hipError_t launch_k(const FusedArgs& a, int n_blocks, hipStream_t s) {
  static_assert(sizeof(Smem<K, TM, R, NW, DR, NM>) <= 160 * 1024, "tile state exceeds the 160 KB LDS of a CU");
  const size_t smem = sizeof(Smem<K, TM, R, NW, DR, NM>);
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_fused<K, TM, R, NW, DR, NM, MODE>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(smem));
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  k_fused<K, TM, R, NW, DR, NM, MODE><<<dim3(unsigned(n_blocks)), dim3(64 * NW), smem, s>>>(a);
  return hipGetLastError();
}

template <int K, int TM, typename R, int NW, int DR, int NM>
hipError_t launch_mode(int mode, const FusedArgs& a, int n_blocks, hipStream_t s) {
  switch (mode) {
    case kCached: return launch_k<K, TM, R, NW, DR, NM, kCached>(a, n_blocks, s);
    case kRecompute: return launch_k<K, TM, R, NW, DR, NM, kRecompute>(a, n_blocks, s);
    case kEncode: return launch_k<K, TM, R, NW, DR, NM, kEncode>(a, n_blocks, s);
    case kRegress: return launch_k<K, TM, R, NW, DR, NM, kRegress>(a, n_blocks, s);
    case kDerive: return launch_k<K, TM, R, NW, DR, NM, kDerive>(a, n_blocks, s);
    case kRadial: return launch_k<K, TM, R, NW, DR, NM, kRadial>(a, n_blocks, s);
    case kCachedTileFj: return launch_k<K, TM, R, NW, DR, NM, kCachedTileFj>(a, n_blocks, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

// Angular configurations: 0 = irreducible basis with l_max <= 3 (16 rows,
// 20 monomials), 1 = Cartesian basis with l_max <= 3 (20 rows in two 16-row
// tiles), 2 = irreducible basis with l_max 4 or 5 (up to 36 rows in three
// tiles, 56 monomials of degree <= 5).
int angular_config(int angular, int lmax) { return angular == 1 ? 1 : (lmax > 3 ? 2 : 0); }

void angular_table_shape(int acfg, int* rows, int* cols) {
  *rows = acfg == 0 ? 16 : (acfg == 1 ? 32 : 48);
  *cols = acfg == 2 ? 56 : kMonomials;
}

// Instantiations: k in {16, 32, 64}; float64 with one wavefront per SIMD,
// float32 with two.  Atoms per tile: float64 16, float32 32 (two column
// groups in the head), fewer where the moment would not fit LDS: at k = 64
// 8 (float64) and 16 (float32); l_max 4..5, whose 36-row moment and 6k-wide
// head input grow with k, 16 / 9 / 3 atoms at k = 16 / 32 / 64 in float64
// and 32 / 16 / 11 in float32 (a tile's listed entries are spread evenly
// over the work-group's threads, which rules out 17-19 at k = 32).  The
// other fusion configurations are built for k = 32 with the irreducible
// basis and l_max <= 3.
int fused_tile_max(int k, int precision, int acfg) {
  if (acfg == 1) return precision == 64 ? 16 : 32;
  if (acfg == 2) {
    if (precision == 64) return k == 16 ? 16 : (k == 32 ? 9 : 3);
    return k == 16 ? 32 : (k == 32 ? 16 : 11);
  }
  if (precision == 64) return k == 64 ? 8 : 16;
  return k == 64 ? 16 : 32;
}

hipError_t launch_fused(int k, int precision, int acfg, int mode, const FusedArgs& a, int n_blocks, hipStream_t s) {
  if (mode != kCached && (k != 32 || acfg != 0)) return hipErrorInvalidValue;
  if (acfg == 1 && k != 32) return hipErrorInvalidValue;
  if (precision == 64) {
    if (acfg == 1) return launch_k<32, 16, double, 4, 32, 20, kCached>(a, n_blocks, s);
    if (acfg == 2) {
      switch (k) {
        case 16: return launch_k<16, 16, double, 4, 48, 56, kCached>(a, n_blocks, s);
        case 32: return launch_k<32, 9, double, 4, 48, 56, kCached>(a, n_blocks, s);
        case 64: return launch_k<64, 3, double, 4, 48, 56, kCached>(a, n_blocks, s);
        default: return hipErrorInvalidValue;
      }
    }
    switch (k) {
      case 16: return launch_k<16, 16, double, 4, 16, 20, kCached>(a, n_blocks, s);
      case 32: return launch_mode<32, 16, double, 4, 16, 20>(mode, a, n_blocks, s);
      case 64: return launch_k<64, 8, double, 4, 16, 20, kCached>(a, n_blocks, s);
      default: break;
    }
  } else if (precision == 32) {
    if (acfg == 1) return launch_k<32, 32, float, 8, 32, 20, kCached>(a, n_blocks, s);
    if (acfg == 2) {
      switch (k) {
        case 16: return launch_k<16, 32, float, 8, 48, 56, kCached>(a, n_blocks, s);
        case 32: return launch_k<32, 16, float, 8, 48, 56, kCached>(a, n_blocks, s);
        case 64: return launch_k<64, 11, float, 8, 48, 56, kCached>(a, n_blocks, s);
        default: return hipErrorInvalidValue;
      }
    }
    switch (k) {
      case 16: return launch_k<16, 32, float, 8, 16, 20, kCached>(a, n_blocks, s);
      case 32: return launch_mode<32, 32, float, 8, 16, 20>(mode, a, n_blocks, s);
      case 64: return launch_k<64, 16, float, 8, 16, 20, kCached>(a, n_blocks, s);
      default: break;
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace mlip
