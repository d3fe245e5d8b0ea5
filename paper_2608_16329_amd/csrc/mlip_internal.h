// Internal declarations of the MLIP library: context layout, constants shared
// by host code and kernels, and the host-side launchers of each kernel file.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/mlip.h"

namespace mlip {

// Fused-kernel geometry (gfx950: 64-wide wavefronts, 160 KB LDS per CU).
constexpr int kWaves = 4;                 // wavefronts per work-group (one per SIMD)
constexpr int kThreads = kWaves * 64;     // work-group size
constexpr int kEntCap = 2048;             // longest neighbour row
// Listed entries and chunks one tile of tm atoms can hold.
constexpr int tile_entry_cap(int tm) { return tm * 128 > kEntCap ? tm * 128 : kEntCap; }
constexpr int tile_chunk_cap(int tm) { return tile_entry_cap(tm) / 16 + 16; }
constexpr int kMaxSpecies = 16;
constexpr int kEncWidth = 128;            // encoder hidden width on the GPU path
constexpr int kHeadWidth = 64;            // head hidden width on the GPU path
constexpr int kMaxHidden = 8;             // hidden layers supported on the GPU path
constexpr int kAngRows = 16;              // angular rows, (lmax+1)^2 <= 16
constexpr int kMonomials = 20;            // Cartesian monomials of degree <= 3
// Fixed per-device scratch of mlip_compute_noalloc (MLIP_STATIC_SCRATCH_BYTES):
// block totals and counters in the first 256 bytes, the fused kernel's
// workspace after them.
constexpr size_t kStaticScratchBytes = size_t(256) << 20;
constexpr size_t kStaticScratchHeader = 256;

// Number of values in one packed encoder table (device layout).
inline size_t enc_table_elems(int k, int enc_hidden) {
  return 2 * kEncWidth + size_t(enc_hidden - 1) * (kEncWidth * kEncWidth + kEncWidth) +
         size_t(k) * kEncWidth + k;
}
// Number of values in one packed head table (device layout).
inline size_t head_table_elems(int nin, int reg_hidden) {
  return 2 * size_t(kHeadWidth) * nin + kHeadWidth +
         size_t(reg_hidden - 1) * (2 * kHeadWidth * kHeadWidth + kHeadWidth) + kHeadWidth + 1;
}

// The neighbour list's entries: caller indices (int32), or 16-bit codes.  A
// code names the neighbour by where the builder found it: which of the up to
// 27 cells scanned around the centre's cell (the index ix + 3 iy + 9 iz into
// the per-dimension candidate lists of `nbr_cells`), the neighbour's species
// s, and its place t in the (s, cell) bucket of the sorted order:
//   code = ((9 iz + 3 iy + ix) << (sbits + tbits)) | (s << tbits) | t,
// sbits = bits of C - 1, tbits = 11 - sbits (27 < 2^5).  The caller index is
// perm[start[s ncell + cell] + t].  The builder writes codes when every
// bucket holds at most 2^tbits atoms, int32 indices otherwise.
struct ListView {
  const int32_t* idx32;       // caller indices (null when the list is coded)
  const uint16_t* idx16;      // codes (null when the list holds indices)
  const int32_t* start;       // [C ncell + 1] first sorted slot of each (species, cell) bucket
  const int32_t* perm;        // sorted slot -> caller index
  const int32_t* key;         // caller index -> bucket key s ncell + cell at the last build
  int nc[3];                  // cells per dimension
  int ncell;
  int tbits, sbits;
};

// Arguments of the fused energy/force/virial kernel.
struct FusedArgs {
  const double* pos;          // caller order [n][3]
  const int32_t* types;       // caller order [n] (library copy)
  const int32_t* perm;        // sorted slot -> caller index
  const int64_t* offsets;     // [n+1], rows in sorted order
  ListView list;              // neighbour entries
  // network tables and workspace hold the kernel's arithmetic type
  // (float64 or float32, mlip_hparams.precision)
  const void* enc;            // packed encoder tables
  const void* head;           // packed head tables
  const void* qc;             // [16][20] angular coefficients
  double* energy;             // [n] or null
  double* forces;             // [n][3], zeroed before launch
  double* virial;             // [n][9] or null
  double* totals;             // [10]: E, W (zeroed before launch)
  unsigned long long* counters;  // [0] active pairs (zeroed before launch)
  void* ws;                   // per-block workspace
  long long ws_slot;          // values per block slot
  void* gbuf;                 // [n][(lmax+1) k] by sorted slot: G, then dE/dG (three-kernel and unfused configurations)
  // unfused configuration, radial kernel: per neighbour-list entry the pair
  // vector and distance written by the setup kernel, and the radial features
  // and their r-derivatives it writes
  const double* geo;          // [entries][4]: dx, dy, dz, r (r = -1 beyond the cutoff)
  void* grad;                 // [entries][k]
  void* gprime;               // [entries][k]
  double box[3];
  double inv_box[3];
  double rc, rc2;
  double pi_rc;               // pi / rc (cutoff function argument scale)
  int lrow[8];                // first angular row of each order l, lrow[lmax+1] = d
  long long enc_stride, head_stride;
  int C, enc_cond, reg_cond, lmax, enc_hidden, reg_hidden;
  int tile_atoms;             // atoms per tile (<= fused_tile_max)
  int n_tiles;
  int species_start[kMaxSpecies + 1];  // first sorted slot of each species
  int tile_start[kMaxSpecies + 1];     // first tile of each species
};

// Arguments of the kernels of the unfused configuration (one kernel per
// equation, every intermediate in HBM).  Per-entry arrays are indexed by the
// neighbour-list entry (rows in sorted order), per-atom arrays by sorted
// slot; the network-side arrays hold the arithmetic type (precision).
struct UnfusedArgs {
  const double* pos;          // caller order [n][3]
  const int32_t* perm;        // sorted slot -> caller index
  const int64_t* offsets;     // [n+1]
  ListView list;              // neighbour entries
  const void* qc;             // angular table [16][20], then the row metric [16]
  double* geo;                // [entries][4]: dx, dy, dz, r (r = -1 beyond the cutoff)
  const void* grad;           // [entries][k]  g_rad (written by the radial kernel)
  const void* gprime;         // [entries][k]  dg_rad/dr
  void* gang;                 // [entries][16] g_ang
  void* jang;                 // [entries][16][3] dg_ang/dr_ij
  void* P;                    // [n][16][k] moment
  void* G;                    // [n][(lmax+1) k] descriptor, then dE/dG
  void* W;                    // [n][16][k] dE/dP
  void* U;                    // [entries][k] dE_i/dg_rad
  void* V;                    // [entries][16] dE_i/dg_ang
  double* forces;             // [n][3], zeroed before launch
  double* virial;             // [n][9] or null
  double* totals;             // [10] (entries 1..9 accumulated here)
  double box[3];
  double inv_box[3];
  double rc2;
  int lrow[8];
  int lmax;
  long long n;                // atoms
  long long n_entries;        // listed entries
};

// Arguments of the neighbour-list kernels.
struct NbrGrid {
  double box[3];
  double half[3];
  double cell_scale[3];   // nc / L
  int nc[3];
  int ncell;
  int C;
  double rl2;
};

}  // namespace mlip

struct mlip_ctx {
  mlip_hparams hp{};
  hipStream_t stream = nullptr;
  int device = 0;
  int n_cu = 0;
  std::string err;
  size_t bytes = 0;

  // weights and tables, in the kernel's arithmetic type (elem_bytes each)
  size_t elem_bytes = 8;
  unsigned char* d_enc = nullptr;
  size_t enc_stride = 0;      // values per encoder table
  int n_enc = 0;
  unsigned char* d_head = nullptr;
  size_t head_stride = 0;     // values per head table
  int n_head = 0;
  unsigned char* d_qc = nullptr;
  double* d_inv_mass = nullptr;   // per species, acceleration factor / mass
  bool masses_set = false;

  // atoms and neighbour list
  int64_t n = 0;
  double box[3] = {0, 0, 0};
  bool built = false;
  int64_t cap_atoms = 0;
  int32_t* d_types = nullptr;
  int32_t* d_perm = nullptr;
  int32_t* d_key = nullptr;
  double* d_spos = nullptr;
  int32_t* d_rowcnt = nullptr;
  int64_t* d_offsets = nullptr;
  unsigned char* d_idx = nullptr;   // entries: uint16 codes or int32 indices (list_compact)
  size_t cap_idx = 0;               // bytes
  bool list_compact = false;
  bool force_wide_list = false;     // mlip_set_list_format(MLIP_LIST_INDEX)
  int list_tbits = 0, list_sbits = 0;
  int32_t* d_cell_count = nullptr;
  int32_t* d_cell_start = nullptr;
  size_t cap_keys = 0;
  int64_t* d_scan_tmp = nullptr;
  size_t cap_scan = 0;
  mlip::NbrGrid grid{};
  int species_start[mlip::kMaxSpecies + 1] = {0};
  int64_t n_listed = 0;
  int max_row = 0;
  int64_t n_builds = 0;

  // fused kernel
  unsigned char* d_ws = nullptr;  // workspace, cap_ws bytes
  size_t cap_ws = 0;
  size_t ws_slot = 0;             // values per work-group slot
  double* d_totals = nullptr;               // [16]
  unsigned long long* d_counters = nullptr; // [4]
  int32_t* d_flags = nullptr;               // [4]
  double* d_reduce = nullptr;               // [4] scratch for md reductions
  int tile_atoms = 0;
  int64_t n_tiles = 0;
  int n_blocks = 0;
  int fusion = 0;                   // mlip_fusion
  int scatter = 0;                  // mlip_scatter
  int acfg = 0;                     // angular configuration of the kernel
  int lrow[8] = {0};                // first angular row of each order
  unsigned char* d_gbuf = nullptr;  // G / dE/dG per atom (three-kernel configuration), cap_gbuf bytes
  size_t cap_gbuf = 0;
  unsigned char* d_unf = nullptr;   // intermediates of the unfused configuration, cap_unf bytes
  size_t cap_unf = 0;
};

namespace mlip {

// angular_tables.cpp: coefficients of the angular features (angular 0
// irreducible, 1 Cartesian) as rows over the Cartesian monomials, padded to
// rows x cols, followed by one descriptor weight per row; lrow[l] = first row
// of order l (lrow[lmax+1] = d).
bool build_angular_table(int lmax, int angular, int rows, int cols, std::vector<double>* out, int lrow[8],
                         std::string* err);

// neighbors.hip
hipError_t launch_bin(const double* pos, const int32_t* types, int64_t n, const NbrGrid& g,
                      int32_t* key, int32_t* cell_count, int32_t* flags, hipStream_t s);
hipError_t launch_scatter(const int32_t* key, int64_t n, const int32_t* cell_start, int32_t* fill,
                          int32_t* perm, int32_t* flags, hipStream_t s);
hipError_t launch_sort_segments(const int32_t* cell_start, int64_t nkeys, int32_t* perm, hipStream_t s);
hipError_t launch_gather_sorted(const double* pos, const int32_t* perm, int64_t n, const NbrGrid& g,
                                double* spos, hipStream_t s);
// rows: count pass (fill false) or fill pass writing int32 indices or, with
// tbits > 0, 16-bit codes (ListView) into idx
hipError_t launch_rows(const double* spos, const int32_t* perm, int64_t n, const NbrGrid& g,
                       const int32_t* cell_start, int32_t* rowcnt, const int64_t* offsets, void* idx,
                       int32_t* flags, bool fill, int tbits, int sbits, hipStream_t s);
hipError_t launch_exclusive_scan_i32_to_i32(const int32_t* in, int64_t n, int32_t* out, int64_t* tmp,
                                            hipStream_t s);
hipError_t launch_exclusive_scan_i32_to_i64(const int32_t* in, int64_t n, int64_t* out, int64_t* tmp,
                                            hipStream_t s);
size_t scan_tmp_elems(int64_t n);
hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s);
hipError_t launch_fill_f64(double* p, int64_t n, double v, hipStream_t s);
hipError_t launch_fill_u64(unsigned long long* p, int64_t n, hipStream_t s);

// fused.hip.  k 16, 32 or 64; precision 64 or 32; angular configuration
// acfg 0 (irreducible, l_max <= 3: 16 rows x 20 monomials), 1 (Cartesian,
// l_max <= 3: 32 x 20) or 2 (irreducible, l_max 4..5: 48 x 56); mode 0
// cached, 1 recompute, 2 encoding, 3 regression, 4 derivation kernel of the
// three-kernel split.  Modes other than 0 exist for k = 32 with acfg 0, and
// acfg 1 for k = 32.
int angular_config(int angular, int lmax);
void angular_table_shape(int acfg, int* rows, int* cols);
int fused_tile_max(int k, int precision, int acfg);  // centre atoms per tile of that instantiation
hipError_t launch_fused(int k, int precision, int acfg, int mode, const FusedArgs& a, int n_blocks, hipStream_t s);
// Modes of launch_fused used by the unfused configuration.
constexpr int kModeRegress = 3;   // Eq. 6: G -> E_i, dE/dG
constexpr int kModeRadial = 5;    // Eq. 2: distances -> g_rad, dg_rad/dr per entry
// The cached single kernel with the tile-reduced F_j scatter (k = 32,
// acfg 0): F_j contributions summed per distinct neighbour of a tile in
// LDS, then one global atomic per neighbour.
constexpr int kModeCachedTileFj = 6;

// unfused.hip: the other eight kernels of the unfused configuration, in
// order; k = 32, irreducible basis with l_max <= 3.
enum UnfusedStage { kUnfSetup, kUnfAngular, kUnfMoment, kUnfDescriptor, kUnfAdjoint, kUnfU, kUnfV, kUnfForce };
hipError_t launch_unfused(int stage, int precision, const UnfusedArgs& a, hipStream_t s);

// scratch.hip: the device address of the fixed scratch on `device`, which
// must be the current device; resolved on first use and kept per device.
hipError_t static_scratch_address(int device, void** out);

// md.hip
hipError_t launch_md_first_half(double* pos, double* vel, const double* forces, const int32_t* types,
                                const double* inv_mass, int64_t n, double dt, const double* ref,
                                double* max_disp2, hipStream_t s);
hipError_t launch_md_disp_since_build(const double* pos, const int32_t* perm, const double* spos, int64_t n,
                                     const double box[3], double* max_disp2, hipStream_t s);
hipError_t launch_md_second_half(double* vel, const double* forces, const int32_t* types,
                                 const double* inv_mass, int64_t n, double dt, hipStream_t s);
hipError_t launch_md_kinetic(const double* vel, const int32_t* types, const double* inv_mass, int64_t n,
                             double* out, hipStream_t s);

}  // namespace mlip
