// Host runtime of the C ABI: contexts, weight files, per-precision weight
// packing, graph buffers and the orchestration of the graph and forward
// kernels.  No arithmetic of the model runs here.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <fstream>
#include <new>

#include "internal.h"

namespace {

painn_status fail(painn_ctx* ctx, painn_status st, const std::string& msg) {
  if (ctx) ctx->err = msg;
  return st;
}

painn_status hip_fail(painn_ctx* ctx, hipError_t e, const char* what) {
  return fail(ctx, PAINN_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define HIP_TRY(ctx, expr)                                   \
  do {                                                       \
    hipError_t e_ = (expr);                                  \
    if (e_ != hipSuccess) return hip_fail((ctx), e_, #expr); \
  } while (0)

// Grow a device buffer to hold at least `n` elements (contents not kept).
template <typename T>
hipError_t ensure(T** p, size_t* cap, size_t n) {
  if (n <= *cap && *p) return hipSuccess;
  if (*p) {
    hipError_t e = hipFree(*p);
    if (e != hipSuccess) return e;
    *p = nullptr;
  }
  size_t want = n < 16 ? 16 : n + n / 4;
  hipError_t e = hipMalloc((void**)p, want * sizeof(T));
  if (e != hipSuccess) {
    *cap = 0;
    return e;
  }
  *cap = want;
  return hipSuccess;
}

// Round-to-nearest-even of an FP64 value to bfloat16 (8 significant bits).
bf16_t to_bf16(double x) {
  if (isnan(x)) return 0x7FC0;
  if (x == 0.0) return signbit(x) ? 0x8000 : 0x0000;
  int e;
  double m = frexp(x, &e);                      // x = m 2^e, 0.5 <= |m| < 1
  double r = nearbyint(ldexp(m, 8));            // keep 8 significant bits, ties to even
  float f = (float)ldexp(r, e - 8);             // exact (or inf / subnormal at the range ends)
  uint32_t u;
  memcpy(&u, &f, 4);
  return (bf16_t)(u >> 16);
}

double bf16_value(bf16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

// Value of an FP64 weight after rounding to the precision's storage type.
double stored(double x, int prec) {
  if (prec == PAINN_FP64) return x;
  if (prec == PAINN_FP32) return (double)(float)x;
  return bf16_value(to_bf16(x));
}

size_t elem_bytes(int prec) { return prec == PAINN_FP64 ? 8 : prec == PAINN_FP32 ? 4 : 2; }
size_t acc_bytes(int prec) { return prec == PAINN_FP64 ? 8 : 4; }

// Write `vals` (doubles) to host bytes of the storage type.
void put_storage(std::vector<unsigned char>& out, size_t idx, double x, int prec) {
  if (prec == PAINN_FP64) {
    memcpy(&out[idx * 8], &x, 8);
  } else if (prec == PAINN_FP32) {
    float f = (float)x;
    memcpy(&out[idx * 4], &f, 4);
  } else {
    bf16_t h = to_bf16(x);
    memcpy(&out[idx * 2], &h, 2);
  }
}

void put_acc(std::vector<unsigned char>& out, size_t idx, double x, int prec) {
  if (prec == PAINN_FP64) {
    memcpy(&out[idx * 8], &x, 8);
  } else {
    float f = (float)x;
    memcpy(&out[idx * 4], &f, 4);
  }
}

hipError_t upload(PrecModel* pm, const std::vector<unsigned char>& host, void** dst) {
  hipError_t e = hipMalloc(dst, host.size() ? host.size() : 16);
  if (e != hipSuccess) return e;
  pm->allocs.push_back(*dst);
  if (host.empty()) return hipSuccess;
  return hipMemcpy(*dst, host.data(), host.size(), hipMemcpyHostToDevice);
}

// Pack W [dout][din] (FP64, row-major) and bias [dout] (or null) for `prec`.
// din_p: pad32(din) for a dense layer (filter = 0); MFMA k-blocks of the
// radial filter: filter_kblocks(din, prec) with its bias column (filter = 1),
// filter_kblocks_nb(din, prec) without (filter = 2).
hipError_t pack_dense(PrecModel* pm, int prec, const double* W, const double* b, int dout,
                      int din, DenseDev* out, int filter = 0) {
  // k per MFMA step: BF16 32; FP32 dense layers 16 (4 chained 4-k
  // instructions fed by one 16-byte load per lane), the FP32 filter and FP64 4
  const int KC = prec == PAINN_BF16 ? 32 : prec == PAINN_FP32 && !filter ? 16 : 4;
  const int KPL = KC / 4;
  const int dout_p = pad32(dout);
  const int din_p = filter == 1 ? filter_kblocks(din, prec) * KC
                  : filter == 2 ? filter_kblocks_nb(din, prec) * KC : pad32(din);
  const int nkb = din_p / KC, nct = dout_p / 16;
  std::vector<unsigned char> wh((size_t)dout_p * din_p * elem_bytes(prec), 0);
  for (int ct = 0; ct < nct; ++ct)
    for (int kb = 0; kb < nkb; ++kb)
      for (int l = 0; l < 64; ++l)
        for (int e = 0; e < KPL; ++e) {
          int row = 16 * ct + l % 16, k = KC * kb + KPL * (l / 16) + e;
          double x = (row < dout && k < din) ? W[(size_t)row * din + k] : 0.0;
          size_t idx = (((size_t)ct * nkb + kb) * 64 + l) * KPL + e;
          put_storage(wh, idx, x, prec);
        }
  std::vector<unsigned char> bh((size_t)dout_p * acc_bytes(prec), 0);
  for (int r = 0; r < dout; ++r) put_acc(bh, r, b ? stored(b[r], prec) : 0.0, prec);
  out->din = din;
  out->dout = dout;
  out->din_p = din_p;
  out->dout_p = dout_p;
  hipError_t e = upload(pm, wh, &out->w);
  if (e != hipSuccess) return e;
  return upload(pm, bh, &out->b);
}

void free_prec(PrecModel* pm) {
  if (!pm) return;
  for (void* p : pm->allocs) (void)hipFree(p);
  delete pm;
}

painn_status build_prec(painn_model* m, int prec, PrecModel** out) {
  painn_ctx* ctx = m->ctx;
  const Hyper& hp = m->hp;
  const int F = hp.F, K = hp.K;
  PrecModel* pm = new (std::nothrow) PrecModel();
  if (!pm) return fail(ctx, PAINN_E_OOM, "host allocation failed");
  pm->prec = prec;
  const double* M = m->master.data();
  auto arr = [&](size_t i) { return M + m->offsets[i]; };
  hipError_t e = hipSuccess;
  {
    std::vector<unsigned char> h((size_t)hp.n_species * F * elem_bytes(prec));
    for (size_t i = 0; i < (size_t)hp.n_species * F; ++i) put_storage(h, i, arr(0)[i], prec);
    e = upload(pm, h, &pm->emb);
  }
  pm->layers.resize(hp.L);
  for (int l = 0; l < hp.L && e == hipSuccess; ++l) {
    size_t base = 1 + (size_t)A_PER_LAYER * l;
    LayerDev& L = pm->layers[l];
    e = pack_dense(pm, prec, arr(base + A_PHI_W1), arr(base + A_PHI_B1), F, F, &L.phi1);
    if (e == hipSuccess)
      e = pack_dense(pm, prec, arr(base + A_PHI_W2), arr(base + A_PHI_B2), 3 * F, F, &L.phi2);
    if (e == hipSuccess) {
      std::vector<double> uv((size_t)2 * F * F);
      memcpy(uv.data(), arr(base + A_U), sizeof(double) * F * F);
      memcpy(uv.data() + (size_t)F * F, arr(base + A_V), sizeof(double) * F * F);
      e = pack_dense(pm, prec, uv.data(), nullptr, 2 * F, F, &L.uv);
    }
    if (e == hipSuccess)
      e = pack_dense(pm, prec, arr(base + A_UPD_W1), arr(base + A_UPD_B1), F, 2 * F, &L.upd1);
    if (e == hipSuccess)
      e = pack_dense(pm, prec, arr(base + A_UPD_W2), arr(base + A_UPD_B2), 3 * F, F, &L.upd2);
    if (e == hipSuccess) {
      // [Wf | bf] as one K+1 -> 3F layer; its input row is [f_c g_0 .. f_c g_{K-1}, f_c]
      std::vector<double> wf((size_t)3 * F * (K + 1));
      for (int c = 0; c < 3 * F; ++c) {
        for (int k = 0; k < K; ++k) wf[(size_t)c * (K + 1) + k] = arr(base + A_FILT_W)[(size_t)c * K + k];
        wf[(size_t)c * (K + 1) + K] = arr(base + A_FILT_B)[c];
      }
      if (prec == PAINN_BF16) {
        // BF16 feeds the basis as hi + lo bf16 terms: the layer sees the
        // input [hi | lo] (2K+2 columns) and the filter twice along K.
        std::vector<double> w2((size_t)3 * F * 2 * (K + 1));
        for (int c = 0; c < 3 * F; ++c)
          for (int k = 0; k < 2 * (K + 1); ++k)
            w2[(size_t)c * 2 * (K + 1) + k] = wf[(size_t)c * (K + 1) + k % (K + 1)];
        e = pack_dense(pm, prec, w2.data(), nullptr, 3 * F, 2 * (K + 1), &L.filt_mma, 1);
      } else {
        e = pack_dense(pm, prec, wf.data(), nullptr, 3 * F, K + 1, &L.filt_mma, 1);
      }
    }
    if (e == hipSuccess) {
      // the filter without its bias column, the bias kept beside it (the
      // forward's message where that saves MFMA k-blocks)
      const double* Wf = arr(base + A_FILT_W);
      if (prec == PAINN_BF16) {
        std::vector<double> w2((size_t)3 * F * 2 * K);
        for (int c = 0; c < 3 * F; ++c)
          for (int k = 0; k < 2 * K; ++k) w2[(size_t)c * 2 * K + k] = Wf[(size_t)c * K + k % K];
        e = pack_dense(pm, prec, w2.data(), arr(base + A_FILT_B), 3 * F, 2 * K, &L.filt_nb, 2);
      } else {
        e = pack_dense(pm, prec, Wf, arr(base + A_FILT_B), 3 * F, K, &L.filt_nb, 2);
      }
    }
  }
  size_t idx = 1 + (size_t)A_PER_LAYER * hp.L;
  int din = F;
  for (size_t mm = 0; mm < hp.shared_dims.size() && e == hipSuccess; ++mm) {
    DenseDev d;
    e = pack_dense(pm, prec, arr(idx), arr(idx + 1), hp.shared_dims[mm], din, &d);
    pm->shared.push_back(d);
    din = hp.shared_dims[mm];
    idx += 2;
  }
  pm->branch.resize(hp.n_heads);
  for (int h = 0; h < hp.n_heads && e == hipSuccess; ++h) {
    int di = din;
    for (size_t mm = 0; mm < hp.branch_dims.size() && e == hipSuccess; ++mm) {
      DenseDev d;
      e = pack_dense(pm, prec, arr(idx), arr(idx + 1), hp.branch_dims[mm], di, &d);
      pm->branch[h].push_back(d);
      di = hp.branch_dims[mm];
      idx += 2;
    }
  }
  if (e == hipSuccess) {
    const size_t nb = hp.branch_dims.size();
    std::vector<unsigned char> tab((size_t)hp.n_heads * nb * 2 * sizeof(void*));
    void** tp = (void**)tab.data();
    for (int h = 0; h < hp.n_heads; ++h)
      for (size_t mm = 0; mm < nb; ++mm) {
        tp[(h * nb + mm) * 2] = pm->branch[h][mm].w;
        tp[(h * nb + mm) * 2 + 1] = pm->branch[h][mm].b;
      }
    e = upload(pm, tab, &pm->head_table);
  }
  if (e == hipSuccess && hp.has_blend) {
    int di = hp.n_species;
    std::vector<int> dims = hp.blend_dims;
    dims.push_back(hp.n_heads);
    for (size_t mm = 0; mm < dims.size() && e == hipSuccess; ++mm) {
      DenseDev d;
      e = pack_dense(pm, prec, arr(idx), arr(idx + 1), dims[mm], di, &d);
      pm->blend.push_back(d);
      di = dims[mm];
      idx += 2;
    }
  }
  if (e == hipSuccess && hp.L > 0) {
    // layer 0's phi per species, computed once on the context's stream
    const size_t bytes = (size_t)hp.n_species * 3 * F * elem_bytes(prec);
    e = hipMalloc(&pm->h0, bytes ? bytes : 16);
    if (e == hipSuccess) {
      pm->allocs.push_back(pm->h0);
      e = launch_phi0_table(ctx->stream, prec, F, hp.n_species, pm, pm->h0);
    }
  }
  if (e != hipSuccess) {
    free_prec(pm);
    return hip_fail(ctx, e, "uploading packed weights");
  }
  *out = pm;
  return PAINN_OK;
}

painn_status parse_model(painn_ctx* ctx, const unsigned char* buf, size_t n, painn_model** out) {
  WeightFile wf;
  std::string msg;
  const int st = parse_weight_file(buf, n, &wf, &msg);
  if (st != PAINN_OK) return fail(ctx, (painn_status)st, msg);
  painn_model* m = new (std::nothrow) painn_model();
  if (!m) return fail(ctx, PAINN_E_OOM, "host allocation failed");
  m->ctx = ctx;
  m->hp = std::move(wf.hp);
  m->master.swap(wf.master);
  m->offsets.swap(wf.offsets);
  *out = m;
  return PAINN_OK;
}

}  // namespace

// Workspace of one forward pass, carved in this order: s [N][F], v[0], v[1],
// h [N][3F] (storage type), e [N] (accumulation type), the radial basis rows
// [E + 16][kcols] (storage type), the edge info [E][4] (accumulation type),
// then the head binning: plan (1 KiB), tiles [N M / 16 + 65][4] and the
// (atom, head) order [N M] (int32), with M = 1 entry per atom (one dataset's
// head) or M = H (blended heads); blended heads add the composition
// [B][pad32(S)] (storage type), the head weights [B][H] and the per-head atom
// energies [N][H] (accumulation type).
static size_t head_tiles_bytes(size_t entries) { return (entries / 16 + 65) * 16; }

size_t forward_workspace_bytes(int prec, int N, long long E, int F, int kcols, int B, int H,
                               int S, bool blend) {
  const size_t eb = elem_bytes(prec), ab = acc_bytes(prec);
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t n = (size_t)N, ne = (size_t)E, ent = n * (blend ? (size_t)H : 1);
  size_t b = al(n * F * eb) + 3 * al(n * 3 * F * eb) + al(n * ab) + al((ne + 16) * kcols * eb) +
             al(ne * 4 * ab) + al(1024) + al(head_tiles_bytes(ent)) + al(ent * 4) + al(MSG64_IMAGE_BYTES);
  if (blend) b += al((size_t)B * pad32(S) * eb) + al((size_t)B * H * ab) + al(n * H * ab);
  return b;
}


// ---- per-kernel event timing ------------------------------------------------
struct Profiler {
  bool on = false;
  std::vector<hipEvent_t> pool;
  struct Rec { int kc; hipEvent_t a, b; };
  std::vector<Rec> recs;
  hipEvent_t open[KC_COUNT] = {};
  double ms[KC_COUNT] = {};
  long long launches[KC_COUNT] = {};
};

static const char* kc_name(int kc) {
  static const char* names[KC_COUNT] = {"graph_prep", "graph_count", "graph_scan", "graph_fill",
                                        "embed", "phi", "edge_prep", "message", "update", "heads",
                                        "energy", "export", "transpose", "bwd_heads", "bwd_update",
                                        "bwd_message", "bwd_phi", "force", "train_real", "train_tangent",
                                        "train_adamw"};
  return names[kc];
}

void prof_mark(Profiler* p, hipStream_t s, int kc, bool begin) {
  if (!p || !p->on) return;
  hipEvent_t ev;
  if (p->pool.empty()) {
    if (hipEventCreate(&ev) != hipSuccess) return;
  } else {
    ev = p->pool.back();
    p->pool.pop_back();
  }
  if (hipEventRecord(ev, s) != hipSuccess) {
    p->pool.push_back(ev);
    return;
  }
  if (begin) {
    if (p->open[kc]) p->pool.push_back(p->open[kc]);
    p->open[kc] = ev;
  } else if (p->open[kc]) {
    p->recs.push_back({kc, p->open[kc], ev});
    p->open[kc] = nullptr;
  } else {
    p->pool.push_back(ev);
  }
}

static void prof_collect(Profiler* p) {
  for (auto& r : p->recs) {
    float t = 0.f;
    if (hipEventElapsedTime(&t, r.a, r.b) == hipSuccess) {
      p->ms[r.kc] += t;
      p->launches[r.kc] += 1;
    }
    p->pool.push_back(r.a);
    p->pool.push_back(r.b);
  }
  p->recs.clear();
}

static void prof_free(Profiler* p) {
  if (!p) return;
  for (auto& r : p->recs) { (void)hipEventDestroy(r.a); (void)hipEventDestroy(r.b); }
  for (hipEvent_t e : p->pool) (void)hipEventDestroy(e);
  for (hipEvent_t e : p->open) if (e) (void)hipEventDestroy(e);
  delete p;
}

extern "C" {

const char* painn_status_string(int st) {
  switch (st) {
    case PAINN_OK: return "PAINN_OK";
    case PAINN_E_ARG: return "PAINN_E_ARG";
    case PAINN_E_OOM: return "PAINN_E_OOM";
    case PAINN_E_HIP: return "PAINN_E_HIP";
    case PAINN_E_FILE: return "PAINN_E_FILE";
    case PAINN_E_FORMAT: return "PAINN_E_FORMAT";
    case PAINN_E_SPECIES: return "PAINN_E_SPECIES";
    case PAINN_E_COINCIDENT: return "PAINN_E_COINCIDENT";
    case PAINN_E_UNSUPPORTED: return "PAINN_E_UNSUPPORTED";
    default: return "PAINN_E_UNKNOWN";
  }
}

painn_status painn_create(int device, void* stream, painn_ctx** out) {
  if (!out) return PAINN_E_ARG;
  *out = nullptr;
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || device < 0 || device >= n) return PAINN_E_ARG;
  if (hipSetDevice(device) != hipSuccess) return PAINN_E_HIP;
  painn_ctx* ctx = new (std::nothrow) painn_ctx();
  if (!ctx) return PAINN_E_OOM;
  ctx->device = device;
  ctx->stream = (hipStream_t)stream;
  // the fixed scratch of painn_forward_noalloc: its address on this device
  // (a failed lookup is reported by that entry point, nothing else needs it)
  (void)noalloc_scratch_init(device);
  if (hipHostMalloc((void**)&ctx->h_status, sizeof(DevStatus), hipHostMallocDefault) != hipSuccess) {
    delete ctx;
    return PAINN_E_OOM;
  }
  *out = ctx;
  return PAINN_OK;
}

painn_status painn_set_stream(painn_ctx* ctx, void* stream) {
  if (!ctx) return PAINN_E_ARG;
  ctx->stream = (hipStream_t)stream;
  ctx->err.clear();
  return PAINN_OK;
}

painn_status painn_destroy(painn_ctx* ctx) {
  if (!ctx) return PAINN_OK;
  (void)hipSetDevice(ctx->device);
  (void)hipStreamSynchronize(ctx->stream);
  if (ctx->ws) (void)hipFree(ctx->ws);
  if (ctx->bws) (void)hipFree(ctx->bws);
  if (ctx->h_status) (void)hipHostFree(ctx->h_status);
  prof_free(ctx->prof);
  delete ctx;
  return PAINN_OK;
}

const char* painn_last_error(const painn_ctx* ctx) { return ctx ? ctx->err.c_str() : "null context"; }

painn_status painn_synchronize(painn_ctx* ctx) {
  if (!ctx) return PAINN_E_ARG;
  (void)hipSetDevice(ctx->device);
  HIP_TRY(ctx, hipStreamSynchronize(ctx->stream));
  return PAINN_OK;
}

painn_status painn_model_load_buffer(painn_ctx* ctx, const void* data, size_t nbytes,
                                     painn_model** out) {
  if (!ctx || !data || !out) return fail(ctx, PAINN_E_ARG, "null argument");
  *out = nullptr;
  ctx->err.clear();
  return parse_model(ctx, (const unsigned char*)data, nbytes, out);
}

painn_status painn_model_load(painn_ctx* ctx, const char* path, painn_model** out) {
  if (!ctx || !path || !out) return fail(ctx, PAINN_E_ARG, "null argument");
  *out = nullptr;
  std::ifstream f(path, std::ios::binary);
  if (!f) return fail(ctx, PAINN_E_FILE, std::string("cannot open ") + path);
  std::vector<unsigned char> buf((std::istreambuf_iterator<char>(f)), std::istreambuf_iterator<char>());
  if (f.bad()) return fail(ctx, PAINN_E_FILE, std::string("cannot read ") + path);
  return painn_model_load_buffer(ctx, buf.data(), buf.size(), out);
}

painn_status painn_model_options(const painn_model* m, int32_t* has_blend, int32_t* max_neighbors) {
  if (!m) return PAINN_E_ARG;
  if (has_blend) *has_blend = m->hp.has_blend ? 1 : 0;
  if (max_neighbors) *max_neighbors = m->hp.max_neighbors;
  return PAINN_OK;
}

painn_status painn_model_info(const painn_model* m, int32_t* F, int32_t* K, int32_t* L,
                              int32_t* n_species, int32_t* n_heads, double* cutoff) {
  if (!m) return PAINN_E_ARG;
  if (F) *F = m->hp.F_logical;
  if (K) *K = m->hp.K;
  if (L) *L = m->hp.L;
  if (n_species) *n_species = m->hp.n_species;
  if (n_heads) *n_heads = m->hp.n_heads;
  if (cutoff) *cutoff = m->hp.cutoff;
  return PAINN_OK;
}

painn_status painn_model_free(painn_model* m) {
  if (!m) return PAINN_OK;
  if (m->ctx) {
    (void)hipSetDevice(m->ctx->device);
    (void)hipStreamSynchronize(m->ctx->stream);
  }
  for (PrecModel* pm : m->prec) free_prec(pm);
  delete m;
  return PAINN_OK;
}

painn_status painn_graph_free(painn_graph* g) {
  if (!g) return PAINN_OK;
  if (g->ctx) {
    (void)hipSetDevice(g->ctx->device);
    (void)hipStreamSynchronize(g->ctx->stream);
  }
  void* bufs[] = {g->row_ptr, g->counts, g->col, g->shift, g->recv, g->pos, g->species, g->atom_struct,
                  g->cell, g->sinfo, g->struct_ptr, g->scan_tmp, g->d_status, g->grid, g->bin_of,
                  g->wrap, g->bin_atoms, g->bin_count, g->bin_start, g->bin_scan_tmp,
                  g->counts_cap, g->row_ptr_full, g->col_full, g->shift_full, g->recv_full,
                  g->t_ptr, g->t_edge, g->t_count};
  for (void* p : bufs)
    if (p) (void)hipFree(p);
  delete g;
  return PAINN_OK;
}

painn_status painn_build_graph(painn_ctx* ctx, int32_t B, int32_t N, const int32_t* struct_ptr,
                               const double* pos, const int32_t* species, const double* cell,
                               const uint8_t* pbc, double cutoff, painn_graph** inout) {
  return painn_build_graph_capped(ctx, B, N, struct_ptr, pos, species, cell, pbc, cutoff, 0, inout);
}

painn_status painn_build_graph_capped(painn_ctx* ctx, int32_t B, int32_t N, const int32_t* struct_ptr,
                                      const double* pos, const int32_t* species, const double* cell,
                                      const uint8_t* pbc, double cutoff, int32_t max_neighbors,
                                      painn_graph** inout) {
  if (!ctx) return PAINN_E_ARG;
  ctx->err.clear();
  if (max_neighbors < 0) return fail(ctx, PAINN_E_ARG, "max_neighbors must be >= 0");
  if (!inout) return fail(ctx, PAINN_E_ARG, "inout is null");
  if (B < 0 || N < 0) return fail(ctx, PAINN_E_ARG, "negative size");
  if (B == 0 && N != 0) return fail(ctx, PAINN_E_ARG, "atoms given without structures");
  if (!struct_ptr || (N > 0 && (!pos || !species)))
    return fail(ctx, PAINN_E_ARG, "null input pointer");
  if (pbc && !cell) return fail(ctx, PAINN_E_ARG, "pbc given without cell");
  if (!(cutoff > 0.0) || !isfinite(cutoff)) return fail(ctx, PAINN_E_ARG, "cutoff must be finite and > 0");
  (void)hipSetDevice(ctx->device);
  painn_graph* g = *inout;
  bool fresh = false;
  if (!g) {
    g = new (std::nothrow) painn_graph();
    if (!g) return fail(ctx, PAINN_E_OOM, "host allocation failed");
    g->ctx = ctx;
    fresh = true;
  }
  auto bail = [&](painn_status st, const std::string& msg) {
    if (fresh) painn_graph_free(g);
    return fail(ctx, st, msg);
  };
  // from here on the graph's buffers change: it is unusable until the build
  // completes (a failed rebuild keeps it that way)
  g->valid = false;
  g->t_valid = false;
  g->B = B;
  g->N = N;
  g->cutoff = cutoff;
  g->any_pbc = pbc != nullptr;
  hipError_t e = hipSuccess;
  size_t capa = g->cap_atoms, caps = g->cap_struct, capsc = g->cap_scan;
  // per-atom buffers share one capacity
  if (N + 1 > (long long)g->cap_atoms || !g->row_ptr) {
    size_t c0 = 0, c1 = 0, c2 = 0, c3 = 0, c4 = 0, c5 = 0, c6 = 0, c7 = 0;
    void** old[] = {(void**)&g->row_ptr, (void**)&g->counts, (void**)&g->pos, (void**)&g->species,
                    (void**)&g->atom_struct, (void**)&g->bin_of, (void**)&g->wrap, (void**)&g->bin_atoms};
    for (void** q : old)
      if (*q) { (void)hipFree(*q); *q = nullptr; }
    e = ensure(&g->row_ptr, &c0, (size_t)N + 1);
    if (e == hipSuccess) e = ensure(&g->counts, &c1, c0);
    if (e == hipSuccess) e = ensure(&g->pos, &c2, 3 * c0);
    if (e == hipSuccess) e = ensure(&g->species, &c3, c0);
    if (e == hipSuccess) e = ensure(&g->atom_struct, &c4, c0);
    if (e == hipSuccess) e = ensure(&g->bin_of, &c5, c0);
    if (e == hipSuccess) e = ensure(&g->wrap, &c6, 3 * c0);
    if (e == hipSuccess) e = ensure(&g->bin_atoms, &c7, c0);
    capa = c0;
  }
  if (e == hipSuccess && (B + 1 > (long long)g->cap_struct || !g->sinfo)) {
    size_t c0 = 0, c1 = 0, c2 = 0, c3 = 0;
    if (g->sinfo) { (void)hipFree(g->sinfo); g->sinfo = nullptr; }
    if (g->cell) { (void)hipFree(g->cell); g->cell = nullptr; }
    if (g->struct_ptr) { (void)hipFree(g->struct_ptr); g->struct_ptr = nullptr; }
    if (g->grid) { (void)hipFree(g->grid); g->grid = nullptr; }
    e = ensure(&g->sinfo, &c0, (size_t)B + 1);
    if (e == hipSuccess) e = ensure(&g->cell, &c1, 9 * c0);
    if (e == hipSuccess) e = ensure(&g->struct_ptr, &c2, c0);
    if (e == hipSuccess) e = ensure(&g->grid, &c3, c0);
    caps = c0;
  }
  size_t nblk = ((size_t)N + 1023) / 1024 + 1;
  if (e == hipSuccess) e = ensure(&g->scan_tmp, &capsc, nblk);
  // cell-list bins: structure b owns [2 lo_b + 27 b, 2 hi_b + 27 (b + 1))
  g->n_bins = 2 * (size_t)N + 27 * (size_t)B;
  size_t capb = g->cap_bins, capbs = g->cap_bin_scan;
  if (e == hipSuccess && (g->n_bins + 1 > g->cap_bins || !g->bin_count)) {
    size_t c0 = 0, c1 = 0;
    if (g->bin_count) { (void)hipFree(g->bin_count); g->bin_count = nullptr; }
    if (g->bin_start) { (void)hipFree(g->bin_start); g->bin_start = nullptr; }
    e = ensure(&g->bin_count, &c0, g->n_bins + 1);
    if (e == hipSuccess) e = ensure(&g->bin_start, &c1, c0);
    capb = c0;
  }
  if (e == hipSuccess) e = ensure(&g->bin_scan_tmp, &capbs, (g->n_bins + 1023) / 1024 + 1);
  g->cap_bins = capb;
  g->cap_bin_scan = capbs;
  g->max_neighbors = max_neighbors;
  if (e == hipSuccess && max_neighbors > 0 &&
      ((size_t)N + 1 > g->cap_atoms_cap || !g->row_ptr_full || !g->counts_cap)) {
    size_t c0 = 0, c1 = 0;
    if (g->row_ptr_full) { (void)hipFree(g->row_ptr_full); g->row_ptr_full = nullptr; }
    if (g->counts_cap) { (void)hipFree(g->counts_cap); g->counts_cap = nullptr; }
    g->cap_atoms_cap = 0;
    e = ensure(&g->row_ptr_full, &c0, (size_t)N + 1);
    if (e == hipSuccess) e = ensure(&g->counts_cap, &c1, c0);
    if (e == hipSuccess) g->cap_atoms_cap = c0;
  }
  if (e == hipSuccess && !g->d_status) e = hipMalloc((void**)&g->d_status, sizeof(DevStatus));
  if (e != hipSuccess) return bail(PAINN_E_OOM, std::string("device allocation: ") + hipGetErrorString(e));
  g->cap_atoms = capa;
  g->cap_struct = caps;
  g->cap_scan = capsc;

  (void)hipGetLastError();   // do not report an error left by earlier, unrelated calls
  // with a cap, the full CSR lives in the *_full arrays: a copy of the
  // descriptor points the count/scan/fill launches at them
  painn_graph full = *g;
  if (max_neighbors > 0) full.row_ptr = g->row_ptr_full;
  e = launch_graph_prep(ctx->stream, ctx->prof, B, N, struct_ptr, pos, species, cell, pbc, cutoff, g);
  if (e == hipSuccess) e = launch_graph_count(ctx->stream, ctx->prof, g);
  if (e == hipSuccess) e = launch_graph_scan(ctx->stream, ctx->prof, max_neighbors > 0 ? &full : g);
  if (e == hipSuccess && max_neighbors > 0) e = launch_graph_cap_scan(ctx->stream, ctx->prof, g);
  if (e == hipSuccess)
    e = hipMemcpyAsync(ctx->h_status, g->d_status, sizeof(DevStatus), hipMemcpyDeviceToHost, ctx->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return bail(PAINN_E_HIP, std::string("graph build: ") + hipGetErrorString(e));
  }
  DevStatus st = *ctx->h_status;
  if (st.err) {
    std::string msg;
    painn_status code = PAINN_E_ARG;
    if (st.err & ERR_STRUCT_PTR) msg += "struct_ptr is not a partition of [0, n_atoms); ";
    if (st.err & ERR_CELL) msg += "singular or non-finite periodic cell; ";
    if (st.err & ERR_IMAGES) msg += "periodic image range too large; ";
    if (st.err & ERR_EDGES) msg += "more than 2^31-1 edges; ";
    if (st.err & ERR_COINCIDENT) {
      msg += "coincident atoms (distance 0); ";
      if (!(st.err & ~ERR_COINCIDENT)) code = PAINN_E_COINCIDENT;
    }
    g->E = 0;
    return bail(code, msg);
  }
  g->E_full = st.n_edges;
  g->E = max_neighbors > 0 ? st.n_edges_cap : st.n_edges;
  g->species_min = st.species_min;
  g->species_max = st.species_max;
  if (max_neighbors > 0 && ((size_t)g->E_full > g->cap_edges_full || !g->col_full)) {
    size_t c1 = 0, c2 = 0, c3 = 0;
    if (g->col_full) { (void)hipFree(g->col_full); g->col_full = nullptr; }
    if (g->shift_full) { (void)hipFree(g->shift_full); g->shift_full = nullptr; }
    if (g->recv_full) { (void)hipFree(g->recv_full); g->recv_full = nullptr; }
    e = ensure(&g->col_full, &c1, (size_t)g->E_full);
    if (e == hipSuccess) e = ensure(&g->shift_full, &c2, c1);
    if (e == hipSuccess) e = ensure(&g->recv_full, &c3, c1);
    if (e != hipSuccess) {
      g->cap_edges_full = 0;
      return bail(PAINN_E_OOM, std::string("edge allocation: ") + hipGetErrorString(e));
    }
    g->cap_edges_full = c1;
  }
  size_t cape = g->cap_edges;
  if ((size_t)g->E > g->cap_edges || !g->col) {
    size_t c2 = 0;
    if (g->col) { (void)hipFree(g->col); g->col = nullptr; }
    if (g->shift) { (void)hipFree(g->shift); g->shift = nullptr; }
    if (g->recv) { (void)hipFree(g->recv); g->recv = nullptr; }
    size_t c3 = 0;
    e = ensure(&g->col, &cape, (size_t)g->E);
    if (e == hipSuccess) e = ensure(&g->shift, &c2, cape);
    if (e == hipSuccess) e = ensure(&g->recv, &c3, cape);
    if (e != hipSuccess) {
      g->cap_edges = 0;
      return bail(PAINN_E_OOM, std::string("edge allocation: ") + hipGetErrorString(e));
    }
    g->cap_edges = cape;
  }
  if (max_neighbors > 0) {
    full = *g;
    full.row_ptr = g->row_ptr_full;
    full.col = g->col_full;
    full.shift = g->shift_full;
    full.recv = g->recv_full;
    full.E = g->E_full;
    e = launch_graph_fill(ctx->stream, ctx->prof, &full);
    if (e == hipSuccess) e = launch_graph_cap_select(ctx->stream, ctx->prof, g);
  } else {
    e = launch_graph_fill(ctx->stream, ctx->prof, g);
  }
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return bail(PAINN_E_HIP, std::string("graph fill: ") + hipGetErrorString(e));
  }
  g->valid = true;
  *inout = g;
  return PAINN_OK;
}

painn_status painn_graph_csr(const painn_graph* g, int64_t* n_edges, int32_t* n_atoms,
                             int32_t* n_struct, const int32_t** row_ptr, const int32_t** col,
                             const int32_t** shift) {
  if (!g || !g->valid) return PAINN_E_ARG;
  if (n_edges) *n_edges = g->E;
  if (n_atoms) *n_atoms = g->N;
  if (n_struct) *n_struct = g->B;
  if (row_ptr) *row_ptr = g->row_ptr;
  if (col) *col = g->col;
  if (shift) *shift = g->shift;
  return PAINN_OK;
}

static painn_status run_forward(painn_ctx* ctx, const painn_model* model, const painn_graph* g,
                                const int32_t* dataset_id, painn_precision prec, int stop_layer,
                                double* energies, double* s_out, double* v_out, bool blend = false,
                                double skip = 0.0, double* weights_out = nullptr, void* save = nullptr,
                                ForwardArgs* keep = nullptr, void* ws_fixed = nullptr,
                                size_t ws_fixed_bytes = 0) {
  if (!ctx) return PAINN_E_ARG;
  ctx->err.clear();
  if (!model || !g) return fail(ctx, PAINN_E_ARG, "null model or graph");
  if (model->ctx != ctx || g->ctx != ctx) return fail(ctx, PAINN_E_ARG, "model or graph from another context");
  if (!g->valid) return fail(ctx, PAINN_E_ARG, "graph is not built (its last build failed)");
  if (prec != PAINN_FP64 && prec != PAINN_FP32 && prec != PAINN_BF16)
    return fail(ctx, PAINN_E_ARG, "unknown precision");
  if (g->cutoff != model->hp.cutoff)
    return fail(ctx, PAINN_E_ARG, "graph cutoff differs from the model's cutoff");
  if (g->max_neighbors != model->hp.max_neighbors)
    return fail(ctx, PAINN_E_ARG, "graph neighbour cap differs from the model's");
  if (g->N > 0 && (g->species_min < 0 || g->species_max >= model->hp.n_species))
    return fail(ctx, PAINN_E_SPECIES, "species index outside [0, n_species)");
  (void)hipSetDevice(ctx->device);
  painn_model* m = const_cast<painn_model*>(model);
  if (!m->prec[prec]) {
    if (ws_fixed)
      return fail(ctx, PAINN_E_ARG, "the model's weights are not packed for this precision yet: run "
                                    "painn_forward once at this precision before painn_forward_noalloc");
    painn_status st = build_prec(m, prec, &m->prec[prec]);
    if (st != PAINN_OK) return st;
  }
  const LayerDev& L0 = m->prec[prec]->layers[0];
  const int kcols = L0.filt_mma.din_p > L0.filt_nb.din_p ? L0.filt_mma.din_p : L0.filt_nb.din_p;
  size_t need = forward_workspace_bytes(prec, g->N, g->E, m->hp.F, kcols, g->B, m->hp.n_heads,
                                       m->hp.n_species, blend);
  void* ws = ctx->ws;
  if (ws_fixed) {
    if (need > ws_fixed_bytes)
      return fail(ctx, PAINN_E_ARG, "this batch needs " + std::to_string(need) +
                                        " bytes of workspace; painn_forward_noalloc has " +
                                        std::to_string(ws_fixed_bytes));
    ws = ws_fixed;
  } else if (need > ctx->ws_bytes) {
    if (ctx->ws) {
      (void)hipStreamSynchronize(ctx->stream);
      (void)hipFree(ctx->ws);
      ctx->ws = nullptr;
      ctx->ws_bytes = 0;
    }
    size_t want = need + need / 4;
    hipError_t e = hipMalloc(&ctx->ws, want);
    if (e != hipSuccess) return fail(ctx, PAINN_E_OOM, "forward workspace allocation failed");
    ctx->ws_bytes = want;
    ws = ctx->ws;
  }
  ForwardArgs a{};
  a.m = m;
  a.pm = m->prec[prec];
  a.g = g;
  a.dataset_id = dataset_id;
  a.energies = energies;
  a.stop_layer = stop_layer;
  a.prof = ws_fixed ? nullptr : ctx->prof;   // event timers create events on first use
  a.s_out = s_out;
  a.v_out = v_out;
  a.save = save;
  // carve the workspace
  const size_t eb = elem_bytes(prec), ab = acc_bytes(prec);
  const size_t N = g->N, F = m->hp.F;
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  char* p = (char*)ws;
  a.s = p; p += al(N * F * eb);
  a.v[0] = p; p += al(N * 3 * F * eb);
  a.v[1] = p; p += al(N * 3 * F * eb);
  a.h = p; p += al(N * 3 * F * eb);
  a.e = p; p += al(N * ab);
  a.basis = p; p += al(((size_t)g->E + 16) * kcols * eb);
  a.einfo = p; p += al((size_t)g->E * 4 * ab);
  a.msg_img = p; p += al(MSG64_IMAGE_BYTES);
  const size_t ent = N * (blend ? (size_t)m->hp.n_heads : 1);
  a.head_plan = p; p += al(1024);
  a.head_tiles = p; p += al(head_tiles_bytes(ent));
  a.head_order = (int32_t*)p; p += al(ent * 4);
  a.blend = blend;
  a.skip = skip;
  a.weights_out = weights_out;
  a.comp = a.hw = a.eh = nullptr;
  if (blend) {
    const size_t H = m->hp.n_heads;
    a.comp = p; p += al((size_t)g->B * pad32(m->hp.n_species) * eb);
    a.hw = p; p += al((size_t)g->B * H * ab);
    a.eh = p; p += al(N * H * ab);
  }
  if (keep) *keep = a;
  if (g->B == 0 && !s_out) return PAINN_OK;
  (void)hipGetLastError();   // do not report an error left by earlier, unrelated calls
  hipError_t e = launch_forward(ctx->stream, prec, a);
  if (e != hipSuccess) {
    (void)hipGetLastError();  // leave no sticky error for the caller's next HIP call
    return hip_fail(ctx, e, "forward launch");
  }
  return PAINN_OK;
}

// Reverse-pass workspace: save area, gradients dE/ds, dE/dv (two of each),
// dE/dh, basis rows and their derivatives and edge info in sender order,
// per-edge partials (one slot per wave of the
// channels), per-atom scratch, per-edge dE/dr.
static int forces_scratch_width(const Hyper& hp) {
  int zw = 0;
  const int nl = (int)(hp.shared_dims.size() + hp.branch_dims.size());
  for (int m = 0; m + 1 < nl; ++m)
    zw += pad32(m < (int)hp.shared_dims.size() ? hp.shared_dims[m]
                                               : hp.branch_dims[m - hp.shared_dims.size()]);
  return zw > hp.F ? zw : hp.F;
}

// Operand buffers in global memory, for reverse tile kernels whose 16-row
// tiles do not fit the LDS: [16][3F + pad] per update / phi tile (FP64 at
// F = 384), [2][16][widest head layer + 2] per heads workgroup.
static size_t forces_xbuf_bytes(int prec, const Hyper& hp, int N, bool blend) {
  const size_t eb = elem_bytes(prec), F = hp.F, tiles = ((size_t)N + 15) / 16;
  const size_t head_tiles = ((size_t)N * (blend ? hp.n_heads : 1) + 15) / 16;
  // LDS row padding of the dense kernels' activation tiles (elements)
  const size_t pad = lds_pad(prec);
  size_t x = 0;
  if (16 * (4 * F + 2 * pad) * eb > 160 * 1024) x = tiles * 16 * (3 * F + pad) * eb;
  int wmax = hp.F;
  for (int d : hp.shared_dims) wmax = wmax > pad32(d) ? wmax : pad32(d);
  for (size_t mm = 0; mm + 1 < hp.branch_dims.size(); ++mm)
    wmax = wmax > pad32(hp.branch_dims[mm]) ? wmax : pad32(hp.branch_dims[mm]);
  const size_t hb = (size_t)2 * 16 * (wmax + pad) * eb;
  if (hb > 150 * 1024) {
    const size_t grid = head_tiles + hp.n_heads < (size_t)HB_GRID ? head_tiles + hp.n_heads : (size_t)HB_GRID;
    const size_t h = grid * hb;
    x = x > h ? x : h;
  }
  return x;
}

// per-atom rows, or the reverse heads kernel's 16 rows per workgroup
static size_t forces_scratch_rows(int N) {
  return (size_t)N > (size_t)HB_GRID * 16 ? (size_t)N : (size_t)HB_GRID * 16;
}

static size_t forces_workspace_bytes(int prec, const Hyper& hp, int N, long long E, int kcols, bool blend) {
  const size_t eb = elem_bytes(prec), ab = acc_bytes(prec), n = (size_t)N, F = hp.F;
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  return al(forces_xbuf_bytes(prec, hp, N, blend)) + al(blend ? n * hp.n_heads * F * ab : 0) +
         al(SaveLayout::bytes(n, F, hp.L, eb)) + 2 * al(n * F * ab) + 3 * al(n * 3 * F * ab) +
         2 * al(((size_t)E + 16) * kcols * eb) + al((size_t)E * 4 * ab) + al((size_t)E * (F / 16) * 4 * ab) +
         al(forces_scratch_rows(N) * forces_scratch_width(hp) * ab) + al((size_t)E * 3 * sizeof(double));
}

// Transposed layers for the reverse pass (from the FP64 master weights).
static hipError_t pack_transposed(PrecModel* pm, int prec, const double* W, int dout, int din, DenseDev* out) {
  std::vector<double> t((size_t)dout * din);
  for (int o = 0; o < dout; ++o)
    for (int k = 0; k < din; ++k) t[(size_t)k * dout + o] = W[(size_t)o * din + k];
  return pack_dense(pm, prec, t.data(), nullptr, din, dout, out);
}

static painn_status build_prec_T(painn_model* m, PrecModel* pm) {
  const Hyper& hp = m->hp;
  const int F = hp.F, prec = pm->prec;
  const double* M = m->master.data();
  auto arr = [&](size_t i) { return M + m->offsets[i]; };
  hipError_t e = hipSuccess;
  for (int l = 0; l < hp.L && e == hipSuccess; ++l) {
    const size_t base = 1 + (size_t)A_PER_LAYER * l;
    LayerDev& L = pm->layers[l];
    e = pack_transposed(pm, prec, arr(base + A_PHI_W1), F, F, &L.phi1T);
    if (e == hipSuccess) e = pack_transposed(pm, prec, arr(base + A_PHI_W2), 3 * F, F, &L.phi2T);
    if (e == hipSuccess) {
      // [U^T | V^T]: row o, column k < F -> U[k][o], column F + k -> V[k][o]
      std::vector<double> t((size_t)F * 2 * F);
      for (int o = 0; o < F; ++o)
        for (int k = 0; k < F; ++k) {
          t[(size_t)o * 2 * F + k] = arr(base + A_U)[(size_t)k * F + o];
          t[(size_t)o * 2 * F + F + k] = arr(base + A_V)[(size_t)k * F + o];
        }
      e = pack_dense(pm, prec, t.data(), nullptr, F, 2 * F, &L.uvT);
    }
    if (e == hipSuccess) e = pack_transposed(pm, prec, arr(base + A_UPD_W1), F, 2 * F, &L.upd1T);
    if (e == hipSuccess) e = pack_transposed(pm, prec, arr(base + A_UPD_W2), 3 * F, F, &L.upd2T);
  }
  size_t idx = 1 + (size_t)A_PER_LAYER * hp.L;
  int din = F;
  pm->sharedT.clear();
  for (size_t mm = 0; mm < hp.shared_dims.size() && e == hipSuccess; ++mm) {
    DenseDev d;
    e = pack_transposed(pm, prec, arr(idx), hp.shared_dims[mm], din, &d);
    pm->sharedT.push_back(d);
    din = hp.shared_dims[mm];
    idx += 2;
  }
  pm->branchT.assign(hp.n_heads, {});
  const size_t nb = hp.branch_dims.size();
  for (int h = 0; h < hp.n_heads && e == hipSuccess; ++h) {
    int di = din;
    for (size_t mm = 0; mm < nb && e == hipSuccess; ++mm) {
      DenseDev d;
      if (mm + 1 < nb) e = pack_transposed(pm, prec, arr(idx), hp.branch_dims[mm], di, &d);
      pm->branchT[h].push_back(d);   // the output layer has none
      di = hp.branch_dims[mm];
      idx += 2;
    }
  }
  if (e == hipSuccess) {
    std::vector<unsigned char> tab((size_t)hp.n_heads * nb * 2 * sizeof(void*), 0);
    void** tp = (void**)tab.data();
    for (int h = 0; h < hp.n_heads; ++h)
      for (size_t mm = 0; mm < nb; ++mm) tp[(h * nb + mm) * 2] = pm->branchT[h][mm].w;
    e = upload(pm, tab, &pm->head_tableT);
  }
  if (e != hipSuccess) return hip_fail(m->ctx, e, "uploading transposed weights");
  pm->has_T = true;
  return PAINN_OK;
}

static painn_status forces_impl(painn_ctx* ctx, const painn_model* model, const painn_graph* graph,
                                const int32_t* dataset_id, painn_precision precision, double* energies,
                                double* forces, bool blend, double skip, double* weights) {
  if (!ctx) return PAINN_E_ARG;
  ctx->err.clear();
  if (!model || !graph) return fail(ctx, PAINN_E_ARG, "null model or graph");
  if (!graph->valid) return fail(ctx, PAINN_E_ARG, "graph is not built (its last build failed)");
  if (graph->B > 0 && !energies) return fail(ctx, PAINN_E_ARG, "energies is null");
  if (graph->N > 0 && !forces) return fail(ctx, PAINN_E_ARG, "forces is null");
  if (precision == PAINN_BF16) return fail(ctx, PAINN_E_UNSUPPORTED, "forces run in FP64 or FP32");
  if (precision != PAINN_FP64 && precision != PAINN_FP32) return fail(ctx, PAINN_E_ARG, "unknown precision");
  const Hyper& hp = model->hp;
  const size_t eb = elem_bytes(precision);
  if (graph->B == 0) return PAINN_OK;
  (void)hipSetDevice(ctx->device);
  painn_graph* g = const_cast<painn_graph*>(graph);
  painn_model* m = const_cast<painn_model*>(model);
  // every check of the forward, and the precision's packed weights
  if (g->ctx != ctx || m->ctx != ctx) return fail(ctx, PAINN_E_ARG, "model or graph from another context");
  if (g->cutoff != hp.cutoff) return fail(ctx, PAINN_E_ARG, "graph cutoff differs from the model's cutoff");
  if (g->max_neighbors != hp.max_neighbors)
    return fail(ctx, PAINN_E_ARG, "graph neighbour cap differs from the model's");
  if (!m->prec[precision]) {
    painn_status st = build_prec(m, precision, &m->prec[precision]);
    if (st != PAINN_OK) return st;
  }
  PrecModel* pm = m->prec[precision];
  if (!pm->has_T) {
    painn_status st = build_prec_T(m, pm);
    if (st != PAINN_OK) return st;
  }
  // edges grouped by sender
  if (!g->t_valid) {
    hipError_t e = ensure(&g->t_ptr, &g->cap_t_atoms, (size_t)g->N + 1);
    size_t cc = g->cap_t_atoms;
    if (e == hipSuccess) e = ensure(&g->t_count, &cc, (size_t)g->N + 1);
    if (e == hipSuccess) e = ensure(&g->t_edge, &g->cap_t_edges, (size_t)g->E + 1);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      g->cap_t_atoms = g->cap_t_edges = 0;
      return hip_fail(ctx, e, "edge transpose allocation");
    }
    e = launch_transpose(ctx->stream, ctx->prof, g);
    if (e != hipSuccess) return hip_fail(ctx, e, "edge transpose");
    g->t_valid = true;
  }
  const int kcols = pm->layers[0].filt_mma.din_p;
  const size_t need = forces_workspace_bytes(precision, hp, g->N, g->E, kcols, blend);
  if (need > ctx->bws_bytes) {
    if (ctx->bws) {
      (void)hipStreamSynchronize(ctx->stream);
      (void)hipFree(ctx->bws);
      ctx->bws = nullptr;
      ctx->bws_bytes = 0;
    }
    const size_t want = need + need / 8;
    hipError_t e = hipMalloc(&ctx->bws, want);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return fail(ctx, PAINN_E_OOM, "reverse-pass workspace allocation failed");
    }
    ctx->bws_bytes = want;
  }
  const size_t N = g->N, F = hp.F, ab = acc_bytes(precision);
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  char* p = (char*)ctx->bws;
  BackwardArgs b{};
  b.xbuf_bytes = forces_xbuf_bytes(precision, hp, g->N, blend);
  b.xbuf = p; p += al(b.xbuf_bytes);
  b.g_heads = p; p += al(blend ? N * hp.n_heads * F * ab : 0);
  b.save = p; p += al(SaveLayout::bytes(N, F, hp.L, eb));
  b.gs = p; p += al(N * F * ab);
  b.gs2 = p; p += al(N * F * ab);
  b.gv = p; p += al(N * 3 * F * ab);
  b.gv2 = p; p += al(N * 3 * F * ab);
  b.gh = p; p += al(N * 3 * F * ab);
  b.dbasis = p; p += al(((size_t)g->E + 16) * kcols * eb);
  b.basis_t = p; p += al(((size_t)g->E + 16) * kcols * eb);
  b.einfo_t = p; p += al((size_t)g->E * 4 * ab);
  b.eg = p; p += al((size_t)g->E * (F / 16) * 4 * ab);
  b.scratch_w = forces_scratch_width(hp);
  b.scratch = p; p += al(forces_scratch_rows(g->N) * b.scratch_w * ab);
  b.gr = (double*)p;
  ForwardArgs fa{};
  painn_status st = run_forward(ctx, model, graph, dataset_id, precision, hp.L - 1, energies, nullptr, nullptr,
                                blend, skip, weights, b.save, &fa);
  if (st != PAINN_OK) return st;
  b.m = m;
  b.pm = pm;
  b.g = g;
  b.dataset_id = dataset_id;
  b.einfo = fa.einfo;
  b.head_plan = fa.head_plan;
  b.head_tiles = fa.head_tiles;
  b.head_order = fa.head_order;
  b.forces = forces;
  b.blend = blend;
  b.skip = skip;
  b.hw = fa.hw;
  b.prof = ctx->prof;
  (void)hipGetLastError();
  hipError_t e = launch_backward(ctx->stream, precision, b);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return hip_fail(ctx, e, "reverse pass launch");
  }
  return PAINN_OK;
}

painn_status painn_forces(painn_ctx* ctx, const painn_model* model, const painn_graph* graph,
                          const int32_t* dataset_id, painn_precision precision, double* energies,
                          double* forces) {
  return forces_impl(ctx, model, graph, dataset_id, precision, energies, forces, false, 0.0, nullptr);
}

painn_status painn_forces_blend(painn_ctx* ctx, const painn_model* model, const painn_graph* graph,
                                painn_precision precision, double skip_threshold, double* energies,
                                double* forces, double* weights) {
  if (!ctx) return PAINN_E_ARG;
  if (!model || !graph) return fail(ctx, PAINN_E_ARG, "null model or graph");
  if (!model->hp.has_blend)
    return fail(ctx, PAINN_E_UNSUPPORTED, "the model has no branch-weighting MLP");
  if (!(skip_threshold >= 0.0) || !isfinite(skip_threshold))
    return fail(ctx, PAINN_E_ARG, "skip_threshold must be finite and >= 0");
  return forces_impl(ctx, model, graph, nullptr, precision, energies, forces, true, skip_threshold, weights);
}

painn_status painn_forward(painn_ctx* ctx, const painn_model* model, const painn_graph* graph,
                           const int32_t* dataset_id, painn_precision precision, double* energies) {
  if (ctx && graph && graph->B > 0 && !energies) return fail(ctx, PAINN_E_ARG, "energies is null");
  return run_forward(ctx, model, graph, dataset_id, precision, model ? model->hp.L - 1 : 0,
                     energies, nullptr, nullptr);
}

painn_status painn_forward_noalloc(painn_ctx* ctx, const painn_model* model, const painn_graph* graph,
                                   const int32_t* dataset_id, painn_precision precision, double* energies) {
  if (!ctx) return PAINN_E_ARG;
  if (graph && graph->B > 0 && !energies) return fail(ctx, PAINN_E_ARG, "energies is null");
  void* scratch = noalloc_scratch(ctx->device);
  if (!scratch) return fail(ctx, PAINN_E_HIP, "the fixed scratch's device address is not available");
  return run_forward(ctx, model, graph, dataset_id, precision, model ? model->hp.L - 1 : 0, energies,
                     nullptr, nullptr, false, 0.0, nullptr, nullptr, nullptr, scratch,
                     NOALLOC_SCRATCH_BYTES);
}

painn_status painn_forward_blend(painn_ctx* ctx, const painn_model* model, const painn_graph* graph,
                                 painn_precision precision, double skip_threshold, double* energies,
                                 double* weights) {
  if (!ctx) return PAINN_E_ARG;
  if (!model || !graph) return fail(ctx, PAINN_E_ARG, "null model or graph");
  if (!model->hp.has_blend)
    return fail(ctx, PAINN_E_UNSUPPORTED, "the model has no branch-weighting MLP");
  if (!(skip_threshold >= 0.0) || !isfinite(skip_threshold))
    return fail(ctx, PAINN_E_ARG, "skip_threshold must be finite and >= 0");
  if (graph->B > 0 && !energies) return fail(ctx, PAINN_E_ARG, "energies is null");
  return run_forward(ctx, model, graph, nullptr, precision, model->hp.L - 1, energies, nullptr, nullptr,
                     true, skip_threshold, weights);
}

painn_status painn_forward_features(painn_ctx* ctx, const painn_model* model,
                                    const painn_graph* graph, painn_precision precision,
                                    int32_t layer, double* s_out, double* v_out) {
  if (!ctx) return PAINN_E_ARG;
  if (!model || !graph) return fail(ctx, PAINN_E_ARG, "null model or graph");
  if (layer < -1 || layer >= model->hp.L) return fail(ctx, PAINN_E_ARG, "layer out of range");
  if (graph->N > 0 && (!s_out || !v_out)) return fail(ctx, PAINN_E_ARG, "null output");
  return run_forward(ctx, model, graph, nullptr, precision, layer, nullptr, s_out, v_out);
}

painn_status painn_profile_enable(painn_ctx* ctx, int enable) {
  if (!ctx) return PAINN_E_ARG;
  ctx->err.clear();
  if (!ctx->prof) {
    ctx->prof = new (std::nothrow) Profiler();
    if (!ctx->prof) return fail(ctx, PAINN_E_OOM, "host allocation failed");
  }
  ctx->prof->on = enable != 0;
  return PAINN_OK;
}

painn_status painn_profile_read(painn_ctx* ctx, int32_t n_max, const char** names, double* ms,
                                int64_t* launches, int32_t* n_out) {
  if (!ctx || n_max < 0 || (n_max > 0 && (!names || !ms || !launches)) || !n_out)
    return fail(ctx, PAINN_E_ARG, "bad profile_read arguments");
  ctx->err.clear();
  *n_out = 0;
  if (!ctx->prof) return PAINN_OK;
  (void)hipSetDevice(ctx->device);
  HIP_TRY(ctx, hipStreamSynchronize(ctx->stream));
  prof_collect(ctx->prof);
  int n = 0;
  for (int k = 0; k < KC_COUNT && n < n_max; ++k) {
    if (!ctx->prof->launches[k]) continue;
    names[n] = kc_name(k);
    ms[n] = ctx->prof->ms[k];
    launches[n] = ctx->prof->launches[k];
    ++n;
  }
  for (int k = 0; k < KC_COUNT; ++k) { ctx->prof->ms[k] = 0; ctx->prof->launches[k] = 0; }
  *n_out = n;
  return PAINN_OK;
}

}  // extern "C"

