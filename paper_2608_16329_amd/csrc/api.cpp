// C ABI of the MLIP library (declared in include/mlip.h): argument checks,
// weight repacking into MFMA fragment order, device buffers, and the launch
// sequence of the neighbour builder and the fused kernel.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "kernel_math.h"
#include "mlip_internal.h"

using namespace mlip;

namespace {

constexpr double kAccPerForceMass = 9.648533212e-3;  // (eV/A)/amu -> A/fs^2

mlip_status fail(mlip_ctx* ctx, mlip_status st, const std::string& msg) {
  if (ctx) ctx->err = msg;
  return st;
}

// Why the last mlip_create on this thread failed (there is no context to
// hold it); mlip_last_error(NULL) returns it.
thread_local std::string t_create_err;

mlip_status create_fail(mlip_status st, const std::string& msg) {
  t_create_err = msg;
  return st;
}

mlip_status fail_hip(mlip_ctx* ctx, hipError_t e, const char* what) {
  (void)hipGetLastError();
  return fail(ctx, MLIP_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define MLIP_HIP(ctx, expr)                                  \
  do {                                                       \
    const hipError_t e_ = (expr);                            \
    if (e_ != hipSuccess) return fail_hip((ctx), e_, #expr); \
  } while (0)

#define MLIP_TRY(expr)                    \
  do {                                    \
    const mlip_status s_ = (expr);        \
    if (s_ != MLIP_OK) return s_;         \
  } while (0)

template <typename T>
mlip_status ensure(mlip_ctx* ctx, T** p, size_t* cap, size_t need, const char* what) {
  if (*p && need <= *cap) return MLIP_OK;
  if (*p) {
    (void)hipFree(*p);
    ctx->bytes -= *cap * sizeof(T);
    *p = nullptr;
    *cap = 0;
  }
  if (need == 0) return MLIP_OK;
  const hipError_t e = hipMalloc(reinterpret_cast<void**>(p), need * sizeof(T));
  if (e != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    return fail(ctx, MLIP_E_OOM, std::string("device allocation failed: ") + what);
  }
  *cap = need;
  ctx->bytes += need * sizeof(T);
  return MLIP_OK;
}

template <typename T>
void release(mlip_ctx* ctx, T** p, size_t cap) {
  if (*p) {
    (void)hipFree(*p);
    ctx->bytes -= cap * sizeof(T);
    *p = nullptr;
  }
}

bool structurally_valid(const mlip_hparams* hp) {
  return hp && hp->n_species >= 1 && hp->k >= 1 && hp->lmax >= 0 && hp->enc_width >= 1 &&
         hp->enc_hidden >= 1 && hp->reg_width >= 1 && hp->reg_hidden >= 1 && hp->enc_cond >= 0 &&
         hp->enc_cond <= 2 && hp->reg_cond >= 0 && hp->reg_cond <= 1 && (hp->angular == 0 || hp->angular == 1);
}

bool gpu_supported(const mlip_hparams* hp, std::string* why) {
  if (hp->precision != 64 && hp->precision != 32) return *why = "precision must be 64 or 32", false;
  if (hp->angular == 0 && (hp->lmax < 0 || hp->lmax > 5)) return *why = "lmax must be in 0..5 (irreducible)", false;
  if (hp->angular == 1 && (hp->lmax < 0 || hp->lmax > 3)) return *why = "lmax must be in 0..3 (Cartesian)", false;
  if (hp->angular == 1 && hp->k != 32) return *why = "the Cartesian basis runs with k = 32 only", false;
  if (hp->k != 16 && hp->k != 32 && hp->k != 64) return *why = "k must be 16, 32 or 64 on the GPU path", false;
  if (hp->enc_width != kEncWidth) return *why = "enc_width must be 128 on the GPU path", false;
  if (hp->reg_width != kHeadWidth) return *why = "reg_width must be 64 on the GPU path", false;
  if (hp->enc_hidden < 1 || hp->enc_hidden > kMaxHidden) return *why = "enc_hidden must be in 1..8", false;
  if (hp->reg_hidden < 1 || hp->reg_hidden > kMaxHidden) return *why = "reg_hidden must be in 1..8", false;
  if (hp->n_species < 1 || hp->n_species > kMaxSpecies) return *why = "n_species must be in 1..16", false;
  if (!(hp->cutoff > 0.0) || !std::isfinite(hp->cutoff)) return *why = "cutoff must be positive", false;
  if (!(hp->skin >= 0.0) || !std::isfinite(hp->skin)) return *why = "skin must be non-negative", false;
  return true;
}

size_t enc_tables(const mlip_hparams* hp) {
  const size_t C = size_t(hp->n_species);
  return hp->enc_cond == 2 ? C * C : (hp->enc_cond == 1 ? C : 1);
}

size_t head_tables(const mlip_hparams* hp) { return hp->reg_cond == 1 ? size_t(hp->n_species) : 1; }

size_t enc_blob_doubles(const mlip_hparams* hp) {
  const size_t W = size_t(hp->enc_width), k = size_t(hp->k);
  return 2 * W + size_t(hp->enc_hidden - 1) * (W * W + W) + k * W + k;
}

size_t head_blob_doubles(const mlip_hparams* hp) {
  const size_t R = size_t(hp->reg_width), nin = size_t(hp->lmax + 1) * size_t(hp->k);
  return R * nin + R + size_t(hp->reg_hidden - 1) * (R * R + R) + R + 1;
}

// Fragment order of a row-major [nout][nin] matrix for MFMA 16x16x4.  The
// fragment of block (T, i) and output tile t holds, at lane 16 g + c,
// element [16 t + c][16 T + kin(i, g)]; kin is the row map of the MFMA
// result registers (4 i + g for float64, 4 g + i for float32), so that a
// result tile feeds the next product as its B operand.  Fragments of vw
// consecutive output tiles are interleaved per lane so that one 16-byte load
// per lane fetches vw of them: element (T, i, t, lane) sits at
// ((((4 T + i) (nout/16/vw) + t/vw) 64 + lane) vw + t%vw.
void pack_fragments(const double* M, int nout, int nin, int precision, int vw, std::vector<double>* out) {
  const int nt = nout / 16;
  for (int T = 0; T < nin / 16; ++T)
    for (int i = 0; i < 4; ++i)
      for (int u = 0; u < nt / vw; ++u)
        for (int lane = 0; lane < 64; ++lane)
          for (int v = 0; v < vw; ++v) {
            const int g = lane >> 4, c = lane & 15, t = u * vw + v;
            const int kin = precision == 64 ? 4 * i + g : 4 * g + i;
            out->push_back(M[size_t(16 * t + c) * nin + 16 * T + kin]);
          }
}

// Copy host values to the device in the kernel's arithmetic type.
hipError_t upload(void* dev, const double* host, size_t n, size_t elem_bytes) {
  if (elem_bytes == sizeof(double)) return hipMemcpy(dev, host, n * sizeof(double), hipMemcpyHostToDevice);
  std::vector<float> f(n);
  for (size_t i = 0; i < n; ++i) f[i] = float(host[i]);
  return hipMemcpy(dev, f.data(), n * sizeof(float), hipMemcpyHostToDevice);
}

std::vector<double> transpose(const double* M, int rows, int cols) {
  std::vector<double> t(size_t(rows) * cols);
  for (int r = 0; r < rows; ++r)
    for (int c = 0; c < cols; ++c) t[size_t(c) * rows + r] = M[size_t(r) * cols + c];
  return t;
}

// The neighbour list as the kernels read it (ListView).
ListView list_view(const mlip_ctx* ctx) {
  ListView v{};
  v.idx32 = ctx->list_compact ? nullptr : reinterpret_cast<const int32_t*>(ctx->d_idx);
  v.idx16 = ctx->list_compact ? reinterpret_cast<const uint16_t*>(ctx->d_idx) : nullptr;
  v.start = ctx->d_cell_start;
  v.perm = ctx->d_perm;
  v.key = ctx->d_key;
  for (int d = 0; d < 3; ++d) v.nc[d] = ctx->grid.nc[d];
  v.ncell = ctx->grid.ncell;
  v.tbits = ctx->list_tbits;
  v.sbits = ctx->list_sbits;
  return v;
}

// Host copies of what decoding coded entries needs (bucket starts,
// permutation, keys), and a ListView over them.
struct HostList {
  std::vector<int32_t> start, perm, key;
  ListView view{};
};

mlip_status host_list(mlip_ctx* ctx, HostList* h) {
  h->view = list_view(ctx);
  h->view.idx32 = nullptr;
  h->view.idx16 = nullptr;
  if (!ctx->list_compact) return MLIP_OK;
  const size_t n = size_t(ctx->n), nkeys = size_t(ctx->grid.ncell) * size_t(ctx->hp.n_species) + 1;
  h->start.resize(nkeys);
  h->perm.resize(n);
  h->key.resize(n);
  MLIP_HIP(ctx, hipMemcpy(h->start.data(), ctx->d_cell_start, nkeys * sizeof(int32_t), hipMemcpyDeviceToHost));
  MLIP_HIP(ctx, hipMemcpy(h->perm.data(), ctx->d_perm, n * sizeof(int32_t), hipMemcpyDeviceToHost));
  MLIP_HIP(ctx, hipMemcpy(h->key.data(), ctx->d_key, n * sizeof(int32_t), hipMemcpyDeviceToHost));
  h->view.start = h->start.data();
  h->view.perm = h->perm.data();
  h->view.key = h->key.data();
  return MLIP_OK;
}

// Caller indices of entries [beg, beg + len) of the row of caller atom i,
// from a host copy of those entries (int32 or codes).
void decode_row(const mlip_ctx* ctx, const HostList& h, int64_t i, const unsigned char* entries, int64_t len,
                int32_t* out) {
  if (!ctx->list_compact) {
    std::memcpy(out, entries, size_t(len) * sizeof(int32_t));
    return;
  }
  int cand[9];
  centre_cells(h.view, h.key[size_t(i)], cand);
  const uint16_t* codes = reinterpret_cast<const uint16_t*>(entries);
  for (int64_t e = 0; e < len; ++e) out[e] = h.view.perm[code_slot(h.view, cand, codes[e])];
}

// Copy the totals to the host when asked (synchronising the stream).
mlip_status finish_compute(mlip_ctx* ctx, const double* d_totals, double* totals_host) {
  if (totals_host) {
    MLIP_HIP(ctx, hipMemcpyAsync(totals_host, d_totals, 10 * sizeof(double), hipMemcpyDeviceToHost, ctx->stream));
    MLIP_HIP(ctx, hipStreamSynchronize(ctx->stream));
  }
  return MLIP_OK;
}

// The fused kernel's per-work-group workspace, held only in the
// configurations whose kernels park (m, dm) in it (cached, and the
// derivation kernel of the three-kernel split); sized by the last build.
mlip_status ensure_workspace(mlip_ctx* ctx) {
  if (ctx->fusion == MLIP_FUSION_CACHED || ctx->fusion == MLIP_FUSION_PARTIAL)
    return ensure(ctx, &ctx->d_ws, &ctx->cap_ws, ctx->ws_slot * size_t(ctx->n_blocks) * ctx->elem_bytes, "workspace");
  release(ctx, &ctx->d_ws, ctx->cap_ws);
  ctx->cap_ws = 0;
  return MLIP_OK;
}

// Where one evaluation keeps its block totals, active-pair counter and
// fused-kernel workspace: the context's buffers (mlip_compute) or the fixed
// device scratch (mlip_compute_noalloc).
struct ComputeScratch {
  double* totals;                 // [16]
  unsigned long long* counters;   // [4]
  unsigned char* ws;              // ws_slot x n_blocks values
};

// The unfused configuration: ten kernels, one per equation, with the
// per-entry and per-atom intermediates carved out of one device buffer
// (each 256-byte aligned).  a is the fused kernel's argument block with the
// descriptor buffer set.
mlip_status compute_unfused(mlip_ctx* ctx, FusedArgs& a) {
  hipStream_t s = ctx->stream;
  const size_t eb = ctx->elem_bytes, E = size_t(ctx->n_listed), n = size_t(ctx->n);
  const size_t k = size_t(ctx->hp.k), D = kAngRows;
  auto al = [](size_t b) { return (b + 255) / 256 * 256; };
  const size_t sz[9] = {al(4 * sizeof(double) * E), al(k * eb * E), al(k * eb * E), al(D * eb * E),
                        al(3 * D * eb * E), al(D * k * eb * n), al(D * k * eb * n), al(k * eb * E),
                        al(D * eb * E)};
  size_t total = 0;
  for (size_t b : sz) total += b;
  MLIP_TRY(ensure(ctx, &ctx->d_unf, &ctx->cap_unf, total, "unfused intermediates"));
  unsigned char* p[9];
  size_t off = 0;
  for (int i = 0; i < 9; ++i) {
    p[i] = ctx->d_unf + off;
    off += sz[i];
  }
  UnfusedArgs u{};
  u.pos = a.pos;
  u.perm = ctx->d_perm;
  u.offsets = ctx->d_offsets;
  u.list = list_view(ctx);
  u.qc = ctx->d_qc;
  u.geo = reinterpret_cast<double*>(p[0]);
  u.grad = p[1];
  u.gprime = p[2];
  u.gang = p[3];
  u.jang = p[4];
  u.P = p[5];
  u.W = p[6];
  u.U = p[7];
  u.V = p[8];
  u.G = ctx->d_gbuf;
  u.forces = a.forces;
  u.virial = a.virial;
  u.totals = a.totals;
  for (int d = 0; d < 3; ++d) {
    u.box[d] = a.box[d];
    u.inv_box[d] = a.inv_box[d];
  }
  u.rc2 = a.rc2;
  for (int l = 0; l < 8; ++l) u.lrow[l] = a.lrow[l];
  u.lmax = ctx->hp.lmax;
  u.n = ctx->n;
  u.n_entries = ctx->n_listed;
  a.geo = u.geo;
  a.grad = p[1];
  a.gprime = p[2];
  const int kk = ctx->hp.k, prec = ctx->hp.precision;
  MLIP_HIP(ctx, launch_unfused(kUnfSetup, prec, u, s));                         // Eq. 1
  MLIP_HIP(ctx, launch_fused(kk, prec, ctx->acfg, kModeRadial, a, ctx->n_blocks, s));  // Eq. 2
  MLIP_HIP(ctx, launch_unfused(kUnfAngular, prec, u, s));                       // Eq. 3
  MLIP_HIP(ctx, launch_unfused(kUnfMoment, prec, u, s));                        // Eq. 4
  MLIP_HIP(ctx, launch_unfused(kUnfDescriptor, prec, u, s));                    // Eq. 5
  MLIP_HIP(ctx, launch_fused(kk, prec, ctx->acfg, kModeRegress, a, ctx->n_blocks, s));  // Eq. 6
  MLIP_HIP(ctx, launch_unfused(kUnfAdjoint, prec, u, s));                       // Eq. 7
  MLIP_HIP(ctx, launch_unfused(kUnfU, prec, u, s));                             // Eq. 8
  MLIP_HIP(ctx, launch_unfused(kUnfV, prec, u, s));                             // Eq. 9
  MLIP_HIP(ctx, launch_unfused(kUnfForce, prec, u, s));                         // Eq. 10
  return MLIP_OK;
}

// One evaluation (mlip_compute and mlip_compute_noalloc) with the given
// scratch.  Allocates only in the three-kernel and unfused configurations.
mlip_status run_compute(mlip_ctx* ctx, const double* pos_dev, double* energy_dev, double* forces_dev,
                        double* virial_dev, double* totals_host, const ComputeScratch& sc) {
  hipStream_t s = ctx->stream;
  const int64_t n = ctx->n;
  if (n == 0) {
    if (totals_host)
      for (int k = 0; k < 10; ++k) totals_host[k] = 0.0;
    return MLIP_OK;
  }
  if (!pos_dev || !forces_dev) return fail(ctx, MLIP_E_ARG, "NULL positions or forces");
  MLIP_HIP(ctx, launch_fill_f64(forces_dev, 3 * n, 0.0, s));
  MLIP_HIP(ctx, launch_fill_f64(sc.totals, 16, 0.0, s));
  MLIP_HIP(ctx, launch_fill_u64(sc.counters, 4, s));

  FusedArgs a{};
  a.pos = pos_dev;
  a.types = ctx->d_types;
  a.perm = ctx->d_perm;
  a.offsets = ctx->d_offsets;
  a.list = list_view(ctx);
  a.enc = ctx->d_enc;
  a.head = ctx->d_head;
  a.qc = ctx->d_qc;
  for (int l = 0; l < 8; ++l) a.lrow[l] = ctx->lrow[l];
  a.energy = energy_dev;
  a.forces = forces_dev;
  a.virial = virial_dev;
  a.totals = sc.totals;
  a.counters = sc.counters;
  a.ws = sc.ws;
  a.ws_slot = (long long)ctx->ws_slot;
  for (int d = 0; d < 3; ++d) {
    a.box[d] = ctx->box[d];
    a.inv_box[d] = 1.0 / ctx->box[d];
  }
  a.rc = ctx->hp.cutoff;
  a.rc2 = ctx->hp.cutoff * ctx->hp.cutoff;
  a.pi_rc = M_PI / ctx->hp.cutoff;
  a.enc_stride = (long long)ctx->enc_stride;
  a.head_stride = (long long)ctx->head_stride;
  a.C = ctx->hp.n_species;
  a.enc_cond = ctx->hp.enc_cond;
  a.reg_cond = ctx->hp.reg_cond;
  a.lmax = ctx->hp.lmax;
  a.enc_hidden = ctx->hp.enc_hidden;
  a.reg_hidden = ctx->hp.reg_hidden;
  a.tile_atoms = ctx->tile_atoms;
  a.n_tiles = int(ctx->n_tiles);
  int t = 0;
  for (int sp_i = 0; sp_i <= a.C; ++sp_i) {
    a.species_start[sp_i] = ctx->species_start[sp_i];
    a.tile_start[sp_i] = t;
    if (sp_i < a.C) t += (ctx->species_start[sp_i + 1] - ctx->species_start[sp_i] + ctx->tile_atoms - 1) / ctx->tile_atoms;
  }
  if (ctx->fusion == MLIP_FUSION_PARTIAL || ctx->fusion == MLIP_FUSION_UNFUSED) {
    const size_t need = size_t(n) * size_t((ctx->hp.lmax + 1) * ctx->hp.k) * ctx->elem_bytes;
    MLIP_TRY(ensure(ctx, &ctx->d_gbuf, &ctx->cap_gbuf, need, "descriptor buffer"));
    a.gbuf = ctx->d_gbuf;
  }
  if (ctx->fusion == MLIP_FUSION_UNFUSED && ctx->n_tiles > 0) {
    MLIP_TRY(compute_unfused(ctx, a));
    return finish_compute(ctx, sc.totals, totals_host);
  }
  if (ctx->n_tiles > 0) {
    const int k = ctx->hp.k, prec = ctx->hp.precision;
    if (ctx->fusion == MLIP_FUSION_PARTIAL) {
      MLIP_HIP(ctx, launch_fused(k, prec, ctx->acfg, 2, a, ctx->n_blocks, s));
      MLIP_HIP(ctx, launch_fused(k, prec, ctx->acfg, 3, a, ctx->n_blocks, s));
      MLIP_HIP(ctx, launch_fused(k, prec, ctx->acfg, 4, a, ctx->n_blocks, s));
    } else {
      const int mode = ctx->fusion == MLIP_FUSION_RECOMPUTE ? 1
                       : (ctx->scatter == MLIP_SCATTER_TILE ? kModeCachedTileFj : 0);
      MLIP_HIP(ctx, launch_fused(k, prec, ctx->acfg, mode, a, ctx->n_blocks, s));
    }
  }
  return finish_compute(ctx, sc.totals, totals_host);
}

}  // namespace

extern "C" {

size_t mlip_weight_count(const mlip_hparams* hp) {
  if (!structurally_valid(hp)) return 0;
  return enc_tables(hp) * enc_blob_doubles(hp) + head_tables(hp) * head_blob_doubles(hp);
}

mlip_status mlip_create(const mlip_hparams* hp, const double* weights_host, size_t n_weights, void* hip_stream,
                        mlip_ctx** out) {
  t_create_err.clear();
  if (!out) return create_fail(MLIP_E_ARG, "NULL output pointer");
  *out = nullptr;
  if (!hp || !weights_host) return create_fail(MLIP_E_ARG, "NULL hyper-parameters or weights");
  if (!structurally_valid(hp)) return create_fail(MLIP_E_ARG, "invalid hyper-parameters");
  std::string why;
  if (!gpu_supported(hp, &why)) return create_fail(MLIP_E_ARG, "unsupported on the GPU path: " + why);
  if (n_weights != mlip_weight_count(hp))
    return create_fail(MLIP_E_ARG, "n_weights is " + std::to_string(n_weights) + ", the hyper-parameters need " +
                                       std::to_string(mlip_weight_count(hp)));

  mlip_ctx* ctx = new mlip_ctx();
  ctx->hp = *hp;
  ctx->stream = reinterpret_cast<hipStream_t>(hip_stream);
  if (hipGetDevice(&ctx->device) != hipSuccess ||
      hipDeviceGetAttribute(&ctx->n_cu, hipDeviceAttributeMultiprocessorCount, ctx->device) != hipSuccess) {
    (void)hipGetLastError();
    delete ctx;
    return create_fail(MLIP_E_HIP, "no current HIP device");
  }
  const int k = hp->k;
  const int nin = (hp->lmax + 1) * k;
  ctx->n_enc = int(enc_tables(hp));
  ctx->n_head = int(head_tables(hp));
  ctx->enc_stride = enc_table_elems(k, hp->enc_hidden);
  ctx->head_stride = head_table_elems(nin, hp->reg_hidden);
  ctx->elem_bytes = hp->precision == 64 ? sizeof(double) : sizeof(float);
  const int prec = hp->precision;
  // encoder fragments per 16-byte load: hidden layers (8 output tiles) and
  // output layer (k/16 tiles); the head keeps one fragment per load
  const int vw_hid = int(16 / ctx->elem_bytes);
  const int vw_out = std::min(vw_hid, k / 16);

  // encoder tables -> [w0 b0 | (fragments(W_t) b_t)... | fragments(W_out) b_out]
  std::vector<double> enc;
  enc.reserve(ctx->enc_stride * ctx->n_enc);
  const double* src = weights_host;
  const size_t W = kEncWidth;
  for (int t = 0; t < ctx->n_enc; ++t) {
    const double* p = src + size_t(t) * enc_blob_doubles(hp);
    enc.insert(enc.end(), p, p + 2 * W);
    p += 2 * W;
    for (int h = 1; h < hp->enc_hidden; ++h) {
      pack_fragments(p, kEncWidth, kEncWidth, prec, vw_hid, &enc);
      enc.insert(enc.end(), p + W * W, p + W * W + W);
      p += W * W + W;
    }
    pack_fragments(p, k, kEncWidth, prec, vw_out, &enc);
    enc.insert(enc.end(), p + size_t(k) * W, p + size_t(k) * W + k);
  }
  // head tables -> [frag(A0) | frag(A0^T) | c0 | (frag(A_t) frag(A_t^T) c_t)... | a_out c_out]
  std::vector<double> head;
  head.reserve(ctx->head_stride * ctx->n_head);
  const double* hsrc = src + size_t(ctx->n_enc) * enc_blob_doubles(hp);
  const int R = kHeadWidth;
  for (int t = 0; t < ctx->n_head; ++t) {
    const double* p = hsrc + size_t(t) * head_blob_doubles(hp);
    pack_fragments(p, R, nin, prec, 1, &head);
    pack_fragments(transpose(p, R, nin).data(), nin, R, prec, 1, &head);
    head.insert(head.end(), p + size_t(R) * nin, p + size_t(R) * nin + R);
    p += size_t(R) * nin + R;
    for (int h = 1; h < hp->reg_hidden; ++h) {
      pack_fragments(p, R, R, prec, 1, &head);
      pack_fragments(transpose(p, R, R).data(), R, R, prec, 1, &head);
      head.insert(head.end(), p + R * R, p + R * R + R);
      p += R * R + R;
    }
    head.insert(head.end(), p, p + R + 1);
  }
  ctx->acfg = angular_config(hp->angular, hp->lmax);
  int qrows = 0, qcols = 0;
  angular_table_shape(ctx->acfg, &qrows, &qcols);
  std::vector<double> qc;
  std::string err;
  if (!build_angular_table(hp->lmax, hp->angular, qrows, qcols, &qc, ctx->lrow, &err) ||
      enc.size() != ctx->enc_stride * ctx->n_enc ||
      head.size() != ctx->head_stride * ctx->n_head) {
    delete ctx;
    return create_fail(MLIP_E_ARG, err.empty() ? "weight repacking size mismatch" : "angular table: " + err);
  }
  size_t cap = 0, cap2 = 0, cap3 = 0, cap4 = 0, cap5 = 0, cap6 = 0, cap7 = 0, cap8 = 0;
  mlip_status st = MLIP_OK;
  const size_t eb = ctx->elem_bytes;
  if ((st = ensure(ctx, &ctx->d_enc, &cap, enc.size() * eb, "encoder")) != MLIP_OK ||
      (st = ensure(ctx, &ctx->d_head, &cap2, head.size() * eb, "head")) != MLIP_OK ||
      (st = ensure(ctx, &ctx->d_qc, &cap3, qc.size() * eb, "tables")) != MLIP_OK ||
      (st = ensure(ctx, &ctx->d_totals, &cap4, size_t(16), "totals")) != MLIP_OK ||
      (st = ensure(ctx, &ctx->d_counters, &cap5, size_t(4), "counters")) != MLIP_OK ||
      (st = ensure(ctx, &ctx->d_flags, &cap6, size_t(4), "flags")) != MLIP_OK ||
      (st = ensure(ctx, &ctx->d_reduce, &cap7, size_t(4), "reduce")) != MLIP_OK ||
      (st = ensure(ctx, &ctx->d_inv_mass, &cap8, size_t(kMaxSpecies), "masses")) != MLIP_OK) {
    const std::string msg = ctx->err;
    mlip_destroy(ctx);
    return create_fail(st, msg);
  }
  if (upload(ctx->d_enc, enc.data(), enc.size(), eb) != hipSuccess ||
      upload(ctx->d_head, head.data(), head.size(), eb) != hipSuccess ||
      upload(ctx->d_qc, qc.data(), qc.size(), eb) != hipSuccess) {
    (void)hipGetLastError();
    mlip_destroy(ctx);
    return create_fail(MLIP_E_HIP, "weight upload failed");
  }
  *out = ctx;
  return MLIP_OK;
}

mlip_status mlip_build_neighbors(mlip_ctx* ctx, int64_t n_atoms, const double* pos_dev, const int32_t* types_dev,
                                 const double box_host[3]) {
  if (!ctx) return MLIP_E_ARG;
  ctx->err.clear();
  if (!box_host) return fail(ctx, MLIP_E_ARG, "NULL box");
  if (n_atoms < 0 || n_atoms >= (int64_t(1) << 31)) return fail(ctx, MLIP_E_ARG, "n_atoms outside [0, 2^31)");
  if (n_atoms > 0 && (!pos_dev || !types_dev)) return fail(ctx, MLIP_E_ARG, "NULL argument");
  const double rl = ctx->hp.cutoff + ctx->hp.skin;
  for (int d = 0; d < 3; ++d)
    if (!(box_host[d] > 0.0) || !std::isfinite(box_host[d])) return fail(ctx, MLIP_E_BOX, "box edges must be positive");
  const double lmin = std::min(box_host[0], std::min(box_host[1], box_host[2]));
  if (!(rl <= 0.5 * lmin)) return fail(ctx, MLIP_E_BOX, "cutoff + skin exceeds half the smallest box edge");
  ctx->built = false;
  if (n_atoms == 0) {
    // an empty system: nothing to bin; later calls produce nothing
    ctx->n = 0;
    for (int d = 0; d < 3; ++d) ctx->box[d] = box_host[d];
    for (int i = 0; i <= kMaxSpecies; ++i) ctx->species_start[i] = 0;
    ctx->n_listed = 0;
    ctx->max_row = 0;
    ctx->tile_atoms = 0;
    ctx->n_tiles = 0;
    ctx->built = true;
    ctx->n_builds += 1;
    return MLIP_OK;
  }
  const int64_t n = n_atoms;
  const int C = ctx->hp.n_species;
  hipStream_t s = ctx->stream;

  NbrGrid g{};
  int64_t ncell = 1;
  for (int d = 0; d < 3; ++d) {
    g.box[d] = box_host[d];
    g.half[d] = 0.5 * box_host[d];
    g.nc[d] = int(std::max(1.0, std::floor(box_host[d] / (rl * (1.0 + 1e-9)))));
  }
  // keep the key space proportional to the atom count
  while (int64_t(g.nc[0]) * g.nc[1] * g.nc[2] * C > 4 * n + 4096) {
    int dmax = 0;
    for (int d = 1; d < 3; ++d)
      if (g.nc[d] > g.nc[dmax]) dmax = d;
    g.nc[dmax] = std::max(1, g.nc[dmax] / 2);
  }
  for (int d = 0; d < 3; ++d) g.cell_scale[d] = g.nc[d] / box_host[d];
  ncell = int64_t(g.nc[0]) * g.nc[1] * g.nc[2];
  g.ncell = int(ncell);
  g.C = C;
  g.rl2 = rl * rl;
  const int64_t nkeys = ncell * C;

  size_t cap = size_t(ctx->cap_atoms);
  size_t cap_i32 = cap, cap_perm = cap, cap_key = cap, cap_rc = cap, cap_sp = cap * 3, cap_off = cap ? cap + 1 : 0;
  if (size_t(n) > cap) {
    MLIP_TRY(ensure(ctx, &ctx->d_types, &cap_i32, size_t(n), "types"));
    MLIP_TRY(ensure(ctx, &ctx->d_perm, &cap_perm, size_t(n), "perm"));
    MLIP_TRY(ensure(ctx, &ctx->d_key, &cap_key, size_t(n), "keys"));
    MLIP_TRY(ensure(ctx, &ctx->d_rowcnt, &cap_rc, size_t(n), "row counts"));
    MLIP_TRY(ensure(ctx, &ctx->d_spos, &cap_sp, size_t(3 * n), "sorted positions"));
    MLIP_TRY(ensure(ctx, &ctx->d_offsets, &cap_off, size_t(n + 1), "offsets"));
    ctx->cap_atoms = n;
  }
  size_t cap_keys = ctx->cap_keys, cap_keys2 = ctx->cap_keys;
  MLIP_TRY(ensure(ctx, &ctx->d_cell_count, &cap_keys, size_t(nkeys + 1), "cell counts"));
  MLIP_TRY(ensure(ctx, &ctx->d_cell_start, &cap_keys2, size_t(nkeys + 1), "cell starts"));
  ctx->cap_keys = std::min(cap_keys, cap_keys2);
  const size_t scan_need = std::max(scan_tmp_elems(n), scan_tmp_elems(nkeys));
  MLIP_TRY(ensure(ctx, &ctx->d_scan_tmp, &ctx->cap_scan, scan_need, "scan scratch"));

  MLIP_HIP(ctx, hipMemcpyAsync(ctx->d_types, types_dev, size_t(n) * sizeof(int32_t), hipMemcpyDeviceToDevice, s));
  MLIP_HIP(ctx, launch_fill_i32(ctx->d_cell_count, nkeys + 1, 0, s));
  MLIP_HIP(ctx, launch_fill_i32(ctx->d_flags, 4, 0, s));
  MLIP_HIP(ctx, launch_bin(pos_dev, ctx->d_types, n, g, ctx->d_key, ctx->d_cell_count, ctx->d_flags, s));
  MLIP_HIP(ctx, launch_exclusive_scan_i32_to_i32(ctx->d_cell_count, nkeys, ctx->d_cell_start, ctx->d_scan_tmp, s));
  MLIP_HIP(ctx, launch_fill_i32(ctx->d_cell_count, nkeys + 1, 0, s));
  MLIP_HIP(ctx, launch_scatter(ctx->d_key, n, ctx->d_cell_start, ctx->d_cell_count, ctx->d_perm, ctx->d_flags, s));
  MLIP_HIP(ctx, launch_sort_segments(ctx->d_cell_start, nkeys, ctx->d_perm, s));
  MLIP_HIP(ctx, launch_gather_sorted(pos_dev, ctx->d_perm, n, g, ctx->d_spos, s));
  MLIP_HIP(ctx, launch_rows(ctx->d_spos, ctx->d_perm, n, g, ctx->d_cell_start, ctx->d_rowcnt, nullptr, nullptr,
                            ctx->d_flags, false, 0, 0, s));
  MLIP_HIP(ctx, launch_exclusive_scan_i32_to_i64(ctx->d_rowcnt, n, ctx->d_offsets, ctx->d_scan_tmp, s));

  int64_t total = 0;
  int32_t flags[4] = {0, 0, 0, 0};
  int32_t sp[kMaxSpecies + 1];
  MLIP_HIP(ctx, hipMemcpyAsync(&total, ctx->d_offsets + n, sizeof(int64_t), hipMemcpyDeviceToHost, s));
  MLIP_HIP(ctx, hipMemcpyAsync(flags, ctx->d_flags, sizeof(flags), hipMemcpyDeviceToHost, s));
  for (int sp_i = 0; sp_i <= C; ++sp_i)
    MLIP_HIP(ctx, hipMemcpyAsync(&sp[sp_i], ctx->d_cell_start + int64_t(sp_i) * ncell, sizeof(int32_t),
                                 hipMemcpyDeviceToHost, s));
  MLIP_HIP(ctx, hipStreamSynchronize(s));
  if (flags[0]) return fail(ctx, MLIP_E_TYPE, "species outside [0, n_species) or non-finite position");
  if (flags[1] > kEntCap) return fail(ctx, MLIP_E_NBR_CAP, "a neighbour row is longer than 2048 entries");

  // entries as 16-bit codes (cell choice, species, place in the bucket) when
  // every (species, cell) bucket fits the place field, else int32 indices
  int sbits = 0;
  while ((1 << sbits) < C) ++sbits;
  const int tbits = 11 - sbits;
  ctx->list_compact = !ctx->force_wide_list && flags[2] <= (1 << tbits);
  ctx->list_tbits = ctx->list_compact ? tbits : 0;
  ctx->list_sbits = ctx->list_compact ? sbits : 0;
  const size_t entry_bytes = ctx->list_compact ? sizeof(uint16_t) : sizeof(int32_t);
  size_t need = size_t(std::max<int64_t>(total, 1)) * entry_bytes;
  // 1/32 headroom for later builds: in MD the list length drifts by well under
  // that between rebuilds, and every byte of slack is a byte per entry that
  // the largest system cannot use (the old buffer is freed before the new one
  // is allocated, so growing never holds both)
  if (need > ctx->cap_idx) need = need + need / 32;
  MLIP_TRY(ensure(ctx, &ctx->d_idx, &ctx->cap_idx, need, "neighbour list"));
  MLIP_HIP(ctx, launch_rows(ctx->d_spos, ctx->d_perm, n, g, ctx->d_cell_start, ctx->d_rowcnt, ctx->d_offsets,
                            ctx->d_idx, ctx->d_flags, true, ctx->list_tbits, ctx->list_sbits, s));

  ctx->grid = g;
  ctx->n = n;
  for (int d = 0; d < 3; ++d) ctx->box[d] = box_host[d];
  for (int i = 0; i <= C; ++i) ctx->species_start[i] = sp[i];
  ctx->n_listed = total;
  ctx->max_row = flags[1];

  // fused-kernel tiling and workspace
  const int tm = fused_tile_max(ctx->hp.k, ctx->hp.precision, ctx->acfg);
  const int T = std::max(1, std::min(tm, tile_entry_cap(tm) / std::max(1, ctx->max_row)));
  ctx->tile_atoms = T;
  int64_t tiles = 0;
  for (int sp_i = 0; sp_i < C; ++sp_i) tiles += (int64_t(sp[sp_i + 1] - sp[sp_i]) + T - 1) / T;
  ctx->n_tiles = tiles;
  ctx->n_blocks = int(std::max<int64_t>(1, std::min<int64_t>(tiles, ctx->n_cu)));
  const int64_t chunks = std::min<int64_t>(tile_chunk_cap(tm), (int64_t(T) * ctx->max_row + 15) / 16 + C);
  ctx->ws_slot = size_t(chunks) * 2 * size_t(ctx->hp.k) * 16;
  MLIP_TRY(ensure_workspace(ctx));
  ctx->built = true;
  ctx->n_builds += 1;
  return MLIP_OK;
}

mlip_status mlip_compute(mlip_ctx* ctx, const double* pos_dev, double* energy_dev, double* forces_dev,
                         double* virial_dev, double* totals_host) {
  if (!ctx) return MLIP_E_ARG;
  ctx->err.clear();
  if (!ctx->built) return fail(ctx, MLIP_E_STATE, "mlip_build_neighbors has not been called");
  const ComputeScratch sc{ctx->d_totals, ctx->d_counters, ctx->d_ws};
  return run_compute(ctx, pos_dev, energy_dev, forces_dev, virial_dev, totals_host, sc);
}

mlip_status mlip_compute_noalloc(mlip_ctx* ctx, const double* pos_dev, double* energy_dev, double* forces_dev,
                                 double* virial_dev, double* totals_host) {
  if (!ctx) return MLIP_E_ARG;
  ctx->err.clear();
  if (!ctx->built) return fail(ctx, MLIP_E_STATE, "mlip_build_neighbors has not been called");
  if (ctx->fusion != MLIP_FUSION_CACHED && ctx->fusion != MLIP_FUSION_RECOMPUTE)
    return fail(ctx, MLIP_E_ARG,
                "mlip_compute_noalloc runs the single-kernel configurations only (cached or recompute); the "
                "three-kernel and unfused ones hold per-atom intermediates the library allocates");
  // workspace of the current list: one slot per resident work-group (none
  // when the encoder output is recomputed)
  const size_t ws_bytes =
      ctx->fusion == MLIP_FUSION_CACHED ? ctx->ws_slot * size_t(ctx->n_blocks) * ctx->elem_bytes : 0;
  if (kStaticScratchHeader + ws_bytes > kStaticScratchBytes)
    return fail(ctx, MLIP_E_ARG,
                "the fused kernel's workspace needs " + std::to_string(ws_bytes) + " bytes (" +
                    std::to_string(ctx->n_blocks) + " work-groups x " +
                    std::to_string(ctx->ws_slot * ctx->elem_bytes) + "); the fixed scratch holds " +
                    std::to_string(kStaticScratchBytes - kStaticScratchHeader));
  void* base = nullptr;
  const hipError_t e = static_scratch_address(ctx->device, &base);
  if (e != hipSuccess)
    return fail_hip(ctx, e, "static scratch address (the context's device must be current)");
  unsigned char* b = static_cast<unsigned char*>(base);
  const ComputeScratch sc{reinterpret_cast<double*>(b), reinterpret_cast<unsigned long long*>(b + 128),
                          b + kStaticScratchHeader};
  MLIP_TRY(run_compute(ctx, pos_dev, energy_dev, forces_dev, virial_dev, totals_host, sc));
  // the context's own counter keeps the active-pair count for mlip_get_stats
  if (ctx->n > 0)
    MLIP_HIP(ctx, hipMemcpyAsync(ctx->d_counters, sc.counters, sizeof(unsigned long long), hipMemcpyDeviceToDevice,
                                 ctx->stream));
  return MLIP_OK;
}

mlip_status mlip_get_neighbors(mlip_ctx* ctx, int64_t* offsets_host, int32_t* idx_host) {
  if (!ctx) return MLIP_E_ARG;
  if (!offsets_host || !idx_host) return fail(ctx, MLIP_E_ARG, "NULL argument");
  if (!ctx->built) return fail(ctx, MLIP_E_STATE, "no neighbour list");
  const int64_t n = ctx->n;
  if (n == 0) {
    offsets_host[0] = 0;
    return MLIP_OK;
  }
  const size_t eb = ctx->list_compact ? sizeof(uint16_t) : sizeof(int32_t);
  std::vector<int64_t> off(size_t(n + 1));
  std::vector<int32_t> perm(static_cast<size_t>(n));
  std::vector<unsigned char> ent(size_t(std::max<int64_t>(ctx->n_listed, 1)) * eb);
  MLIP_HIP(ctx, hipStreamSynchronize(ctx->stream));
  MLIP_HIP(ctx, hipMemcpy(off.data(), ctx->d_offsets, off.size() * sizeof(int64_t), hipMemcpyDeviceToHost));
  MLIP_HIP(ctx, hipMemcpy(perm.data(), ctx->d_perm, perm.size() * sizeof(int32_t), hipMemcpyDeviceToHost));
  if (ctx->n_listed > 0)
    MLIP_HIP(ctx, hipMemcpy(ent.data(), ctx->d_idx, size_t(ctx->n_listed) * eb, hipMemcpyDeviceToHost));
  HostList h;
  MLIP_TRY(host_list(ctx, &h));
  std::vector<int64_t> len(size_t(n), 0);
  for (int64_t a = 0; a < n; ++a) len[size_t(perm[size_t(a)])] = off[size_t(a + 1)] - off[size_t(a)];
  offsets_host[0] = 0;
  for (int64_t i = 0; i < n; ++i) offsets_host[i + 1] = offsets_host[i] + len[size_t(i)];
  for (int64_t a = 0; a < n; ++a) {
    const int64_t i = perm[size_t(a)];
    decode_row(ctx, h, i, ent.data() + size_t(off[size_t(a)]) * eb, len[size_t(i)], idx_host + offsets_host[i]);
  }
  return MLIP_OK;
}

mlip_status mlip_get_neighbor_rows(mlip_ctx* ctx, const int64_t* atoms_host, int64_t n_rows, int64_t* counts_host,
                                   int32_t* idx_host, int64_t cap) {
  if (!ctx) return MLIP_E_ARG;
  ctx->err.clear();
  if (n_rows < 0 || cap < 0) return fail(ctx, MLIP_E_ARG, "negative row count or capacity");
  if (n_rows > 0 && (!atoms_host || !counts_host)) return fail(ctx, MLIP_E_ARG, "NULL argument");
  if (cap > 0 && !idx_host) return fail(ctx, MLIP_E_ARG, "NULL argument");
  if (!ctx->built) return fail(ctx, MLIP_E_STATE, "no neighbour list");
  const int64_t n = ctx->n;
  for (int64_t r = 0; r < n_rows; ++r)
    if (atoms_host[r] < 0 || atoms_host[r] >= n) return fail(ctx, MLIP_E_ARG, "atom index outside [0, n)");
  if (n_rows == 0) return MLIP_OK;
  // sorted slot of each requested atom, by one pass over the permutation
  // (slot -> caller index)
  std::vector<int32_t> perm(static_cast<size_t>(n));
  MLIP_HIP(ctx, hipStreamSynchronize(ctx->stream));
  MLIP_HIP(ctx, hipMemcpy(perm.data(), ctx->d_perm, perm.size() * sizeof(int32_t), hipMemcpyDeviceToHost));
  std::vector<int64_t> slot_of(static_cast<size_t>(n), -1);
  std::vector<char> wanted(static_cast<size_t>(n), 0);
  for (int64_t r = 0; r < n_rows; ++r) wanted[size_t(atoms_host[r])] = 1;
  for (int64_t a = 0; a < n; ++a)
    if (wanted[size_t(perm[size_t(a)])]) slot_of[size_t(perm[size_t(a)])] = a;
  int64_t total = 0;
  std::vector<int64_t> beg(static_cast<size_t>(n_rows));
  for (int64_t r = 0; r < n_rows; ++r) {
    int64_t off[2];
    MLIP_HIP(ctx, hipMemcpy(off, ctx->d_offsets + slot_of[size_t(atoms_host[r])], sizeof(off), hipMemcpyDeviceToHost));
    beg[size_t(r)] = off[0];
    counts_host[r] = off[1] - off[0];
    total += counts_host[r];
  }
  if (total > cap) return fail(ctx, MLIP_E_ARG, "the rows do not fit in cap entries");
  // bucket starts for decoding, and each requested atom's key
  HostList h;
  h.view = list_view(ctx);
  if (ctx->list_compact) {
    const size_t nkeys = size_t(ctx->grid.ncell) * size_t(ctx->hp.n_species) + 1;
    h.start.resize(nkeys);
    MLIP_HIP(ctx, hipMemcpy(h.start.data(), ctx->d_cell_start, nkeys * sizeof(int32_t), hipMemcpyDeviceToHost));
    h.view.start = h.start.data();
    h.view.perm = perm.data();
    h.key.assign(size_t(n), 0);
    for (int64_t r = 0; r < n_rows; ++r)
      MLIP_HIP(ctx, hipMemcpy(&h.key[size_t(atoms_host[r])], ctx->d_key + atoms_host[r], sizeof(int32_t),
                              hipMemcpyDeviceToHost));
  }
  const size_t eb = ctx->list_compact ? sizeof(uint16_t) : sizeof(int32_t);
  std::vector<unsigned char> ent;
  int64_t at = 0;
  for (int64_t r = 0; r < n_rows; ++r) {
    const int64_t len = counts_host[r];
    if (len > 0) {
      ent.resize(size_t(len) * eb);
      MLIP_HIP(ctx, hipMemcpy(ent.data(), ctx->d_idx + size_t(beg[size_t(r)]) * eb, size_t(len) * eb,
                              hipMemcpyDeviceToHost));
      decode_row(ctx, h, atoms_host[r], ent.data(), len, idx_host + at);
    }
    at += len;
  }
  return MLIP_OK;
}

mlip_status mlip_set_fusion(mlip_ctx* ctx, int32_t fusion) {
  if (!ctx) return MLIP_E_ARG;
  ctx->err.clear();
  if (fusion != MLIP_FUSION_CACHED && fusion != MLIP_FUSION_RECOMPUTE && fusion != MLIP_FUSION_PARTIAL &&
      fusion != MLIP_FUSION_UNFUSED)
    return fail(ctx, MLIP_E_ARG, "unknown fusion configuration");
  if (fusion != MLIP_FUSION_CACHED && (ctx->hp.k != 32 || ctx->acfg != 0))
    return fail(ctx, MLIP_E_ARG,
                "the recompute, three-kernel and unfused configurations exist for k = 32 and the irreducible "
                "basis with l_max <= 3 only");
  // buffers of a configuration that is left are released
  MLIP_HIP(ctx, hipStreamSynchronize(ctx->stream));
  if (fusion != MLIP_FUSION_UNFUSED) {
    release(ctx, &ctx->d_unf, ctx->cap_unf);
    ctx->cap_unf = 0;
  }
  if (fusion != MLIP_FUSION_PARTIAL && fusion != MLIP_FUSION_UNFUSED) {
    release(ctx, &ctx->d_gbuf, ctx->cap_gbuf);
    ctx->cap_gbuf = 0;
  }
  ctx->fusion = fusion;
  // the workspace follows the configuration (sized by the last build)
  if (ctx->built && ctx->n > 0) MLIP_TRY(ensure_workspace(ctx));
  else if (fusion != MLIP_FUSION_CACHED && fusion != MLIP_FUSION_PARTIAL) MLIP_TRY(ensure_workspace(ctx));
  return MLIP_OK;
}

mlip_status mlip_set_scatter(mlip_ctx* ctx, int32_t scatter) {
  if (!ctx) return MLIP_E_ARG;
  ctx->err.clear();
  if (scatter != MLIP_SCATTER_ATOMIC && scatter != MLIP_SCATTER_TILE)
    return fail(ctx, MLIP_E_ARG, "unknown scatter variant");
  if (scatter == MLIP_SCATTER_TILE && (ctx->hp.k != 32 || ctx->acfg != 0))
    return fail(ctx, MLIP_E_ARG, "the tile-reduced scatter exists for k = 32 and the irreducible basis with "
                                 "l_max <= 3 only");
  ctx->scatter = scatter;
  return MLIP_OK;
}

mlip_status mlip_set_list_format(mlip_ctx* ctx, int32_t format) {
  if (!ctx) return MLIP_E_ARG;
  ctx->err.clear();
  if (format != MLIP_LIST_AUTO && format != MLIP_LIST_INDEX) return fail(ctx, MLIP_E_ARG, "unknown list format");
  ctx->force_wide_list = format == MLIP_LIST_INDEX;
  return MLIP_OK;
}

mlip_status mlip_memory_bytes(const mlip_ctx* ctx, size_t* bytes) {
  if (!ctx || !bytes) return MLIP_E_ARG;
  *bytes = ctx->bytes;
  return MLIP_OK;
}

mlip_status mlip_get_stats(mlip_ctx* ctx, mlip_stats* st) {
  if (!ctx || !st) return MLIP_E_ARG;
  std::memset(st, 0, sizeof(*st));
  unsigned long long active = 0;
  if (ctx->d_counters) {
    MLIP_HIP(ctx, hipMemcpyAsync(&active, ctx->d_counters, sizeof(active), hipMemcpyDeviceToHost, ctx->stream));
    MLIP_HIP(ctx, hipStreamSynchronize(ctx->stream));
  }
  st->n_atoms = ctx->n;
  st->n_listed_pairs = ctx->n_listed;
  st->n_active_pairs = int64_t(active);
  st->max_row = ctx->max_row;
  st->tile_atoms = ctx->tile_atoms;
  st->n_tiles = ctx->n_tiles;
  st->n_blocks = ctx->n_blocks;
  st->n_cells = ctx->grid.ncell;
  st->n_builds = ctx->n_builds;
  st->device_bytes = ctx->bytes;
  st->list_entry_bytes = ctx->n > 0 ? (ctx->list_compact ? 2 : 4) : 0;
  return MLIP_OK;
}

const char* mlip_last_error(const mlip_ctx* ctx) {
  if (!ctx) return t_create_err.c_str();
  return ctx->err.c_str();
}

void mlip_destroy(mlip_ctx* ctx) {
  if (!ctx) return;
  (void)hipDeviceSynchronize();
  void* bufs[] = {ctx->d_enc, ctx->d_head, ctx->d_qc, ctx->d_inv_mass, ctx->d_types, ctx->d_perm,
                  ctx->d_key, ctx->d_spos, ctx->d_rowcnt, ctx->d_offsets, ctx->d_idx, ctx->d_cell_count,
                  ctx->d_cell_start, ctx->d_scan_tmp, ctx->d_ws, ctx->d_totals, ctx->d_counters,
                  ctx->d_flags, ctx->d_reduce, ctx->d_gbuf, ctx->d_unf};
  for (void* p : bufs)
    if (p) (void)hipFree(p);
  (void)hipGetLastError();
  delete ctx;
}

mlip_status mlip_md_set_masses(mlip_ctx* ctx, const double* masses_host) {
  if (!ctx) return MLIP_E_ARG;
  if (!masses_host) return fail(ctx, MLIP_E_ARG, "NULL masses");
  double inv[kMaxSpecies] = {0};
  for (int s = 0; s < ctx->hp.n_species; ++s) {
    if (!(masses_host[s] > 0.0) || !std::isfinite(masses_host[s])) return fail(ctx, MLIP_E_ARG, "masses must be positive");
    inv[s] = kAccPerForceMass / masses_host[s];
  }
  MLIP_HIP(ctx, hipMemcpyAsync(ctx->d_inv_mass, inv, sizeof(inv), hipMemcpyHostToDevice, ctx->stream));
  MLIP_HIP(ctx, hipStreamSynchronize(ctx->stream));
  ctx->masses_set = true;
  return MLIP_OK;
}

mlip_status mlip_md_first_half(mlip_ctx* ctx, double* pos_dev, double* vel_dev, const double* forces_dev, double dt,
                               const double* ref_dev, double* max_disp2_host) {
  if (!ctx) return MLIP_E_ARG;
  if (!ctx->built || !ctx->masses_set) return fail(ctx, MLIP_E_STATE, "build neighbours and set masses first");
  if (ctx->n == 0) {
    if (max_disp2_host) *max_disp2_host = 0.0;
    return MLIP_OK;
  }
  if (!pos_dev || !vel_dev || !forces_dev) return fail(ctx, MLIP_E_ARG, "NULL argument");
  const bool track = max_disp2_host != nullptr;
  if (track) MLIP_HIP(ctx, launch_fill_f64(ctx->d_reduce, 1, 0.0, ctx->stream));
  MLIP_HIP(ctx, launch_md_first_half(pos_dev, vel_dev, forces_dev, ctx->d_types, ctx->d_inv_mass, ctx->n, dt,
                                     track ? ref_dev : nullptr, ctx->d_reduce, ctx->stream));
  if (track && !ref_dev)
    MLIP_HIP(ctx, launch_md_disp_since_build(pos_dev, ctx->d_perm, ctx->d_spos, ctx->n, ctx->box, ctx->d_reduce,
                                             ctx->stream));
  if (track) {
    MLIP_HIP(ctx, hipMemcpyAsync(max_disp2_host, ctx->d_reduce, sizeof(double), hipMemcpyDeviceToHost, ctx->stream));
    MLIP_HIP(ctx, hipStreamSynchronize(ctx->stream));
  }
  return MLIP_OK;
}

mlip_status mlip_md_second_half(mlip_ctx* ctx, double* vel_dev, const double* forces_dev, double dt) {
  if (!ctx) return MLIP_E_ARG;
  if (!ctx->built || !ctx->masses_set) return fail(ctx, MLIP_E_STATE, "build neighbours and set masses first");
  if (ctx->n == 0) return MLIP_OK;
  if (!vel_dev || !forces_dev) return fail(ctx, MLIP_E_ARG, "NULL argument");
  MLIP_HIP(ctx, launch_md_second_half(vel_dev, forces_dev, ctx->d_types, ctx->d_inv_mass, ctx->n, dt, ctx->stream));
  return MLIP_OK;
}

mlip_status mlip_md_kinetic(mlip_ctx* ctx, const double* vel_dev, double* ke_host) {
  if (!ctx) return MLIP_E_ARG;
  if (!ke_host) return fail(ctx, MLIP_E_ARG, "NULL argument");
  if (!ctx->built || !ctx->masses_set) return fail(ctx, MLIP_E_STATE, "build neighbours and set masses first");
  if (ctx->n == 0) {
    *ke_host = 0.0;
    return MLIP_OK;
  }
  if (!vel_dev) return fail(ctx, MLIP_E_ARG, "NULL argument");
  MLIP_HIP(ctx, launch_fill_f64(ctx->d_reduce + 1, 1, 0.0, ctx->stream));
  MLIP_HIP(ctx, launch_md_kinetic(vel_dev, ctx->d_types, ctx->d_inv_mass, ctx->n, ctx->d_reduce + 1, ctx->stream));
  MLIP_HIP(ctx, hipMemcpyAsync(ke_host, ctx->d_reduce + 1, sizeof(double), hipMemcpyDeviceToHost, ctx->stream));
  MLIP_HIP(ctx, hipStreamSynchronize(ctx->stream));
  return MLIP_OK;
}

}  // extern "C"
