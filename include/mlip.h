/*
 * mlip.h - C ABI of the MI355X (gfx950) small-footprint MLIP library.
 *
 * The library evaluates the per-atom energy, forces and virial of the
 * machine-learning interatomic potential of arXiv 2608.16329 (Section 3.1,
 * Eqs. 1-10): for every atom it gathers the neighbours inside the cutoff,
 * builds the species-conditioned radial features (Eq. 2) and the
 * irreducible-harmonic angular features (Eq. 3, Section 3.3), contracts them
 * to the equivariant moment P_i (Eq. 4) and invariant descriptor G_i (Eq. 5),
 * runs the energy head (Eq. 6) and back-propagates analytically to partial
 * forces (Eqs. 7-10).  The MLIP receives coordinates from the MD code and
 * returns energies and forces (Section 2.1, "MLIP Inference").
 *
 * Conventions shared by every call:
 *   - "_dev" pointers are device memory on the context's device (for
 *     example PyTorch-ROCm tensors), contiguous, row-major; "_host" pointers
 *     are host memory.  The caller owns every buffer it passes; the library
 *     never frees or retains caller memory beyond the call, except that
 *     mlip_compute reads the species array given to the last
 *     mlip_build_neighbors from the library's own copy.
 *   - Atom arrays are in the caller's order.  Positions are float64 [n][3]
 *     in Angstrom, species are int32 [n], forces float64 [n][3] in eV/A,
 *     energies float64 [n] in eV, virials float64 [n][9] in eV (row-major
 *     3x3).
 *   - Work is enqueued on the HIP stream given to mlip_create and the call
 *     returns without waiting, unless stated otherwise.
 *   - Every call returns a status; nothing throws or aborts across the ABI.
 *     On failure mlip_last_error(ctx) describes the cause.
 *   - A context is not thread-safe; use one context per host thread.
 *   - Every buffer crossing the ABI is float64 or int32.  The arithmetic of
 *     the network is set by mlip_hparams.precision: 64 evaluates everything
 *     in float64 (Section 4.1); 32 is the reduced-precision mode the paper
 *     evaluates beside it (Sections 3.4 and 4.4), here with the network, the
 *     angular features, the moment/adjoint contractions and the pair
 *     geometry after the minimum-image difference in float32, and that
 *     difference and all force, virial and energy accumulation in float64.
 */
#ifndef MLIP_H
#define MLIP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct mlip_ctx mlip_ctx;

typedef enum {
  MLIP_OK = 0,
  MLIP_E_ARG = -1,      /* NULL pointer, bad size, unsupported hyper-parameter */
  MLIP_E_OOM = -2,      /* device allocation failed                            */
  MLIP_E_HIP = -3,      /* HIP runtime error                                   */
  MLIP_E_BOX = -4,      /* non-positive box edge, or cutoff+skin > min(L)/2    */
  MLIP_E_NBR_CAP = -5,  /* a neighbour row is longer than the kernel can hold  */
  MLIP_E_STATE = -6,    /* call out of order (compute before build_neighbors)  */
  MLIP_E_TYPE = -7      /* species outside [0, n_species) or non-finite input  */
} mlip_status;

/*
 * Hyper-parameters (Section 3.2 species conditioning, Section 3.3 angular
 * basis, Section 4.1 architecture).  Defaults of the paper: k = 32,
 * lmax = 3, irreducible basis, pair-conditioned encoder, species-conditioned
 * head, encoder 3 hidden layers of width 128, head 4 hidden layers of width
 * 64, cutoff 6 A.
 */
typedef struct {
  int32_t n_species;   /* C >= 1 (the GPU path supports C <= 16)                  */
  double  cutoff;      /* r_c in A                                               */
  double  skin;        /* Verlet skin in A; neighbour lists use r_c + skin       */
  int32_t k;           /* radial feature width (GPU path: 16, 32 or 64)          */
  int32_t lmax;        /* maximum angular order (GPU path: 0..5 irreducible,
                          0..3 Cartesian; the Cartesian basis needs k = 32)      */
  int32_t angular;     /* 0 irreducible harmonic basis, d = (lmax+1)^2;
                          1 Cartesian monomials, d = (lmax+1)(lmax+2)(lmax+3)/6,
                          descriptor metric l!/(a!b!c!) (Section 3.3)            */
  int32_t enc_cond;    /* encoder tables: 2 per (s_i,s_j), 1 per s_j, 0 one      */
  int32_t reg_cond;    /* head tables: 1 per s_i, 0 one                          */
  int32_t enc_width;   /* encoder hidden width (GPU path: 128)                   */
  int32_t enc_hidden;  /* encoder hidden layers (GPU path: 1..8)                 */
  int32_t reg_width;   /* head hidden width (GPU path: 64)                       */
  int32_t reg_hidden;  /* head hidden layers (GPU path: 1..8)                    */
  int32_t precision;   /* 64 (float64) or 32 (float32 network, see above)         */
} mlip_hparams;

/* Statistics of the context (mlip_get_stats). */
typedef struct {
  int64_t n_atoms;          /* atoms of the last neighbour build                 */
  int64_t n_listed_pairs;   /* directed pairs within cutoff + skin              */
  int64_t n_active_pairs;   /* directed pairs within cutoff at the last compute */
  int32_t max_row;          /* longest neighbour row                             */
  int32_t tile_atoms;       /* centre atoms per work-group tile                  */
  int64_t n_tiles;          /* tiles of the fused kernel                         */
  int32_t n_blocks;         /* resident work-groups of the fused kernel          */
  int32_t n_cells;          /* cells of the neighbour grid                       */
  int64_t n_builds;         /* neighbour builds so far                           */
  size_t  device_bytes;     /* device memory held by the context                 */
  int32_t list_entry_bytes; /* bytes per neighbour-list entry: 2 (coded), 4      */
} mlip_stats;

/*
 * Number of float64 values in the packed weight blob for these
 * hyper-parameters; 0 if the hyper-parameters are invalid.
 *
 * Blob layout (row-major, matrices [out][in], W = enc_width, R = reg_width):
 *   encoder tables, tau = s_i*C + s_j (enc_cond 2), s_j (1) or 0 (0), each
 *     w0[W] b0[W], then for t = 1..enc_hidden-1: W_t[W][W] b_t[W],
 *     then W_out[k][W] b_out[k]
 *   head tables, rho = s_i (reg_cond 1) or 0, each
 *     A0[R][(lmax+1)*k] c0[R], then for t = 1..reg_hidden-1: A_t[R][R] c_t[R],
 *     then a_out[R] c_out[1]
 * Encoder: h = silu(w0 r + b0); h += silu(W_t h + b_t); g = fc(r) (W_out h +
 * b_out) with fc(r) = (1 + cos(pi r / r_c)) / 2 (Eq. 2).  Head: y =
 * silu(A0 x + c0); y += silu(A_t y + c_t); E_i = a_out . y + c_out (Eq. 6)
 * with x = vec(G_i) in l-major order (index l*k + c).
 */
size_t mlip_weight_count(const mlip_hparams* hp);

/*
 * Create a context on the current HIP device.  Copies and repacks the
 * weights (weights_host, n_weights float64 values, layout above) into device
 * memory, rounded to float32 when precision is 32, and builds the angular
 * projection tables.  hip_stream is a
 * hipStream_t (NULL = default stream); all later work is enqueued on it.
 * Errors: MLIP_E_ARG (bad hparams, unsupported on the GPU path, n_weights
 * mismatch, NULL pointers), MLIP_E_OOM, MLIP_E_HIP.  On error *out is NULL
 * and mlip_last_error(NULL) says why.
 */
mlip_status mlip_create(const mlip_hparams* hp, const double* weights_host, size_t n_weights,
                        void* hip_stream, mlip_ctx** out);

/*
 * Build the neighbour list (Section 3.1: N(i) = atoms within the cutoff;
 * here within cutoff + skin so the list stays valid while atoms move less
 * than skin/2).  Definition (exact, reproducible bit for bit): coordinates
 * wrapped into [0, L) by w = fmod(x, L), +L if negative, -L if >= L; pair
 * vector dx = w_j - w_i folded once by -L if dx > L/2 or +L if dx < -L/2;
 * d2 = (dx*dx + dy*dy) + dz*dz without fused multiply-add; j != i is listed
 * iff d2 < (cutoff + skin)^2.  Rows are grouped by neighbour species.
 * Entries take 2 bytes each (the neighbour's place among the cells scanned
 * around the centre's cell, its species and its place in that cell's
 * species bucket) when every (species, cell) bucket of the cell grid holds at
 * most 2^(11 - ceil(log2 C)) atoms, 4 bytes (its index) otherwise or when
 * mlip_set_list_format asks for indices; mlip_get_stats reports which.
 *   n_atoms   number of atoms (>= 0, < 2^31).  0 records an empty system
 *             (the pointers may then be NULL): later calls succeed and
 *             produce nothing, totals and kinetic energy 0
 *   pos_dev   float64 [n_atoms][3], any real values (wrapped internally)
 *   types_dev int32 [n_atoms], species in [0, n_species); copied
 *   box_host  float64 [3], orthorhombic periodic box edges L_x, L_y, L_z
 * Synchronises the stream (the list length sizes the allocation).
 * Errors: MLIP_E_ARG, MLIP_E_BOX, MLIP_E_TYPE (bad species or non-finite
 * position), MLIP_E_NBR_CAP (a row longer than 2048), MLIP_E_OOM, MLIP_E_HIP.
 */
mlip_status mlip_build_neighbors(mlip_ctx* ctx, int64_t n_atoms, const double* pos_dev,
                                 const int32_t* types_dev, const double box_host[3]);

/*
 * Evaluate energies, forces and virial at pos_dev (float64 [n][3], same n as
 * the last build; atoms must have moved less than skin/2 since then) in one
 * fused pass per atom tile (Eqs. 1-10) that keeps every intermediate on chip
 * except the per-pair radial features, which stay in a fixed-size
 * per-work-group workspace.  Outputs are overwritten:
 *   energy_dev  float64 [n] per-atom E_i, or NULL
 *   forces_dev  float64 [n][3] F_i = -dE/dr_i (required)
 *   virial_dev  float64 [n][9] per-atom w_i = -sum_j r_ij (x) f_ij with
 *               r_ij = r_j - r_i, f_ij = dE_i/dr_ij (row-major), or NULL
 *   totals_host float64 [10] = (E, W[0..8]) summed over atoms, or NULL; when
 *               non-NULL the call synchronises the stream.
 * Errors: MLIP_E_ARG, MLIP_E_STATE (no build), MLIP_E_HIP.
 */
mlip_status mlip_compute(mlip_ctx* ctx, const double* pos_dev, double* energy_dev,
                         double* forces_dev, double* virial_dev, double* totals_host);

/*
 * mlip_compute without device allocation, for callers that cannot allocate:
 * code under HIP graph capture, tight serving loops, hosts that forbid
 * hipMalloc after set-up.  Same arguments, evaluation and outputs as
 * mlip_compute in the single-kernel configurations (MLIP_FUSION_CACHED,
 * MLIP_FUSION_RECOMPUTE).  The fused kernel's per-work-group workspace, the
 * block totals and the active-pair counter go to a fixed scratch array of
 * MLIP_STATIC_SCRATCH_BYTES built into the library, one per device, which
 * that device holds from the first call on it until the process ends; no
 * allocating routine is called.
 *
 * Every call on one device shares that device's scratch and leaves its
 * contents there (the totals and the counter are cleared at the start of a
 * call, the workspace is written before it is read): calls that overlap on
 * one device, from any context or stream, race and give wrong results.
 * Serialise them.  The context's device must be current.
 *
 * Errors: those of mlip_compute; MLIP_E_ARG when the configuration is
 * MLIP_FUSION_PARTIAL or MLIP_FUSION_UNFUSED (they keep per-atom
 * intermediates the library allocates) or when the workspace of the current
 * neighbour list (resident work-groups x per-work-group slot) exceeds the
 * scratch (mlip_last_error gives both sizes); MLIP_E_HIP when the scratch
 * cannot be resolved on the current device.
 */
#define MLIP_STATIC_SCRATCH_BYTES (256u * 1024u * 1024u)
mlip_status mlip_compute_noalloc(mlip_ctx* ctx, const double* pos_dev, double* energy_dev,
                                 double* forces_dev, double* virial_dev, double* totals_host);

/*
 * Copy the neighbour list to the host in caller order: offsets_host int64
 * [n+1], idx_host int32 [offsets[n]] (use mlip_get_stats().n_listed_pairs to
 * size it).  Entries of a row are grouped by neighbour species.  Synchronises.
 */
mlip_status mlip_get_neighbors(mlip_ctx* ctx, int64_t* offsets_host, int32_t* idx_host);

/*
 * Copy the neighbour rows of selected atoms to the host (for checks of the
 * list at sizes where the whole list is too large to copy; the rows are the
 * same as those of mlip_get_neighbors).
 *   atoms_host  int64 [n_rows], caller indices in [0, n), any order, repeats
 *               allowed
 *   counts_host int64 [n_rows], receives the length of each row
 *   idx_host    int32 [cap], receives the rows back to back in the order of
 *               atoms_host (caller indices, grouped by neighbour species)
 * Errors: MLIP_E_ARG (NULL pointer, index outside [0, n), or the rows do not
 * fit in cap entries: counts_host is filled even then), MLIP_E_STATE (no
 * build), MLIP_E_HIP.  Synchronises the stream.
 */
mlip_status mlip_get_neighbor_rows(mlip_ctx* ctx, const int64_t* atoms_host, int64_t n_rows, int64_t* counts_host,
                                   int32_t* idx_host, int64_t cap);

/*
 * Fusion configuration of mlip_compute (Section 3.4, Table "Configurable
 * fusion"); all four give the same results up to rounding.
 *   MLIP_FUSION_CACHED     one kernel: pass 1 keeps the encoder output and its
 *                          radial derivative per pair in a fixed-size
 *                          per-work-group workspace until pass 2 (default)
 *   MLIP_FUSION_RECOMPUTE  one kernel: pass 2 recomputes the encoder (the
 *                          paper's mega-fusion); no workspace traffic, twice
 *                          the encoder work
 *   MLIP_FUSION_PARTIAL    three kernels (Eqs. 1-5; Eq. 6; Eqs. 7-10, the
 *                          paper's partial fusion): G_i and then dE/dG_i go
 *                          through HBM, (l_max+1) k values per atom, which the
 *                          context allocates at the next mlip_compute
 *   MLIP_FUSION_UNFUSED    ten kernels, one per equation of Eqs. 1-10 (the
 *                          table's "before fusion" row): every intermediate
 *                          goes through HBM, per listed neighbour-list entry
 *                          the pair vector and distance, g_rad and dg_rad/dr,
 *                          g_ang and its Jacobian, and the U and V rows
 *                          (4 float64 + 176 values at k = 32), per atom P_i,
 *                          W_i and G_i / dE/dG_i (1152 values at k = 32,
 *                          l_max = 3); allocated at the next mlip_compute
 *                          (MLIP_E_OOM if they do not fit)
 * Values are float64 or float32 as set by mlip_hparams.precision.
 */
typedef enum {
  MLIP_FUSION_CACHED = 0,
  MLIP_FUSION_RECOMPUTE = 1,
  MLIP_FUSION_PARTIAL = 2,
  MLIP_FUSION_UNFUSED = 3
} mlip_fusion;

/*
 * Select the fusion configuration for later mlip_compute calls.  The
 * configurations other than MLIP_FUSION_CACHED exist for k = 32 with the
 * irreducible basis and l_max <= 3.  Synchronises the stream, releases the
 * buffers of a configuration that is left and, after a neighbour build,
 * allocates the per-work-group workspace of the cached and three-kernel
 * configurations (MLIP_E_OOM if it does not fit); the recompute and unfused
 * configurations hold none.
 * Errors: MLIP_E_ARG (unknown value, or a non-default one with other
 * hyper-parameters), MLIP_E_OOM, MLIP_E_HIP.
 */
mlip_status mlip_set_fusion(mlip_ctx* ctx, int32_t fusion);

/*
 * How the cached single kernel adds -f_ij to F_j (Section 3.1: the forces are
 * the scatter-sum of the partial forces), for measuring the two designs
 * against each other; both give the same forces up to rounding order.
 *   MLIP_SCATTER_ATOMIC  one float64 atomic add to HBM per pair and
 *                        component (default)
 *   MLIP_SCATTER_TILE    contributions summed per distinct neighbour of a
 *                        tile in an LDS table, then one atomic add per
 *                        neighbour and component
 * Applies to MLIP_FUSION_CACHED at k = 32 with the irreducible basis and
 * l_max <= 3 (the other configurations scatter by atomics).  Errors:
 * MLIP_E_ARG (unknown value, or MLIP_SCATTER_TILE with other
 * hyper-parameters).
 */
typedef enum { MLIP_SCATTER_ATOMIC = 0, MLIP_SCATTER_TILE = 1 } mlip_scatter;
mlip_status mlip_set_scatter(mlip_ctx* ctx, int32_t scatter);

/*
 * Encoding of the neighbour list's entries from the next mlip_build_neighbors
 * on: MLIP_LIST_AUTO (default) codes entries in 2 bytes whenever the cell
 * grid's buckets allow it, MLIP_LIST_INDEX always stores 4-byte indices.
 * Both give the same neighbour sets and results.  Errors: MLIP_E_ARG.
 */
typedef enum { MLIP_LIST_AUTO = 0, MLIP_LIST_INDEX = 1 } mlip_list_format;
mlip_status mlip_set_list_format(mlip_ctx* ctx, int32_t format);

/* Device memory held by the context, in bytes. */
mlip_status mlip_memory_bytes(const mlip_ctx* ctx, size_t* bytes);

/* Fill *stats (synchronises to read the active-pair counter). */
mlip_status mlip_get_stats(mlip_ctx* ctx, mlip_stats* stats);

/*
 * Text of the last error on this context (never NULL; "" when none).  With
 * ctx NULL: why the last mlip_create on the calling thread failed ("" if it
 * succeeded).
 */
const char* mlip_last_error(const mlip_ctx* ctx);

/* Release the context and its device memory (NULL is ignored). */
void mlip_destroy(mlip_ctx* ctx);

/*
 * Molecular-dynamics driver helpers (velocity Verlet in metal units: A, fs,
 * amu, eV; acceleration = F/m * 9.648533212e-3).  They are not part of the
 * potential; the paper runs its MLIP inside LAMMPS with a 1 fs step
 * (Section 4.1).  They use the species of the last neighbour build.
 */

/* Per-species masses in amu, masses_host float64 [n_species] (> 0). */
mlip_status mlip_md_set_masses(mlip_ctx* ctx, const double* masses_host);

/*
 * First half of a step: vel += dt/2 * a(F); pos += dt * vel.  If
 * max_disp2_host is non-NULL the largest squared displacement is written
 * there (synchronises): against ref_dev (float64 [n][3]) when it is non-NULL,
 * otherwise against the positions of the last neighbour build (minimum image,
 * no extra memory).
 */
mlip_status mlip_md_first_half(mlip_ctx* ctx, double* pos_dev, double* vel_dev,
                               const double* forces_dev, double dt, const double* ref_dev,
                               double* max_disp2_host);

/* Second half of a step: vel += dt/2 * a(F). */
mlip_status mlip_md_second_half(mlip_ctx* ctx, double* vel_dev, const double* forces_dev, double dt);

/* Kinetic energy sum_i m_i |v_i|^2 / 2 in eV into *ke_host (synchronises). */
mlip_status mlip_md_kinetic(mlip_ctx* ctx, const double* vel_dev, double* ke_host);

#ifdef __cplusplus
}
#endif

#endif /* MLIP_H */
