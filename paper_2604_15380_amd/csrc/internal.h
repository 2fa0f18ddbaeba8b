// Internal declarations shared by the host runtime and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "painn.h"
#include "weightfile.h"

typedef uint16_t bf16_t;  // bfloat16 storage (upper half of an IEEE float)

// ---- error bits written by the graph kernels into DevStatus::err ----------
enum : int32_t {
  ERR_STRUCT_PTR = 1,   // struct_ptr not a partition of [0, N)
  ERR_CELL = 2,         // singular or non-finite periodic cell
  ERR_IMAGES = 4,       // image range beyond +-127 or n_atoms*n_images >= 2^31
  ERR_COINCIDENT = 8,   // d2 == 0 for a pair other than (i, i, 0)
  ERR_EDGES = 16,       // more than 2^31 - 1 edges
};

struct DevStatus {      // read back once per build_graph
  long long n_edges;
  int32_t err;
  int32_t species_min;
  int32_t species_max;
  int32_t cells;        // structures searched with a cell list
  long long n_edges_cap;  // edges kept under a neighbour cap
};

struct StructInfo {     // per structure: atom range and periodic image range
  int32_t lo, n;
  int32_t m0, m1, m2;   // |n_k| <= m_k
  int32_t nimg;         // (2 m0 + 1)(2 m1 + 1)(2 m2 + 1)
  // periodic structures: fractional coordinate k of x is x . fr[3k..3k+2];
  // the atoms' fractional range [fmin_k, fmax_k] and r_c / w_k (w_k the
  // cell's width normal to the other two cell vectors), which bound the
  // image shifts one receiver can need
  double fr[9];
  double fmin[3], fmax[3], rw[3];
};

// Cell-list binning of one structure (nb[0] == 0: every pair is tested).
// Bins are at least r_c wide, so every neighbour of an atom lies in the 27
// bins around its own.  Molecules bin Cartesian coordinates over their
// bounding box; periodic cells (all three axes periodic, >= 3 bins each) bin
// the wrapped fractional coordinates.
struct CellGrid {
  int32_t nb[3];
  int32_t base;         // first bin of the structure in the batch's bin arrays
  int32_t periodic;
  int32_t pad;
  double o[3];          // molecules: bin coordinate u_k = (x_k - o_k) s_k
  double s[3];          // periodic:  u_k = (f_k - floor f_k) s_k
  double fr[9];         // periodic:  fractional coordinates f_k = x . fr_k
};

// ---- dense-layer packing ---------------------------------------------------
// A dense layer W [dout, din] is stored padded to (pad32(dout), pad32(din))
// with zeros, in the operand order of a 16x16xKC MFMA: block (ct, kb) holds 64
// lanes x KPL consecutive elements, lane l carrying
// W[16 ct + l % 16][KC kb + KPL (l / 16) + e], e < KPL.
// (FP64/FP32: KC = 4, KPL = 1; BF16: KC = 32, KPL = 8.)
inline __host__ __device__ int pad32(int d) { return (d + 31) & ~31; }

// MFMA k-blocks of the radial filter's input (K+1 basis columns, or 2(K+1)
// for BF16), rounded up to the counts the message kernel is compiled for
// (the padding columns are zero); -1 if too large.
// LDS row padding (elements) of the dense kernels' activation tiles (one
// A-fragment read of 16 rows falls in distinct banks).  The device layouts
// and the host's buffer sizing share it.
constexpr int LDS_PAD_FP64 = 1, LDS_PAD_FP32 = 4, LDS_PAD_BF16 = 8;
inline int lds_pad(int prec) {
  return prec == PAINN_FP64 ? LDS_PAD_FP64 : prec == PAINN_FP32 ? LDS_PAD_FP32 : LDS_PAD_BF16;
}

inline int filter_kblocks(int din, int prec) {
  const int kc = prec == PAINN_BF16 ? 32 : 4;
  const int need = (din + kc - 1) / kc;
  static const int f[] = {3, 6, 9, 12, 17};
  static const int b[] = {1, 2, 3, 5};
  if (prec == PAINN_BF16) {
    for (int x : b) if (need <= x) return x;
  } else {
    for (int x : f) if (need <= x) return x;
  }
  return -1;
}

// The same for the filter without its bias column (K inputs, or 2K for
// BF16): the forward adds f_c b_f in the message's epilogue instead.  Counts
// the message kernel is compiled for in that form; -1 if too large.
inline int filter_kblocks_nb(int din, int prec) {
  const int kc = prec == PAINN_BF16 ? 32 : 4;
  const int need = (din + kc - 1) / kc;
  static const int f[] = {1, 2, 5, 8, 12, 17};
  static const int b[] = {1, 2, 3, 5};
  if (prec == PAINN_BF16) {
    for (int x : b) if (need <= x) return x;
  } else {
    for (int x : f) if (need <= x) return x;
  }
  return -1;
}

struct DenseDev {       // one packed layer on the device
  void* w = nullptr;    // packed weights, storage type of the precision
  void* b = nullptr;    // bias [pad32(dout)], accumulation type (zero padded)
  int din = 0, dout = 0, din_p = 0, dout_p = 0;
};

struct LayerDev {       // one interaction layer
  DenseDev phi1, phi2;  // F -> F (silu), F -> 3F
  DenseDev uv;          // [U; V] stacked: F -> 2F
  DenseDev upd1, upd2;  // 2F -> F (silu), F -> 3F
  DenseDev filt_mma;    // radial filter as a dense layer K+1 -> 3F for MFMA:
                        // input column K is the bias (multiplied by f_c), din
                        // padded to a multiple of the MFMA K step only; BF16
                        // stores it twice along K (input [hi | lo] terms)
  DenseDev filt_nb;     // the filter K -> 3F without the bias column (BF16:
                        // 2K, twice along K), its bias b_f in .b; used by the
                        // energy forward when it needs fewer MFMA k-blocks
                        // (the reverse pass keeps filt_mma)
  // transposed weights for the reverse pass (no bias; built on the first
  // forces call): phi1^T F -> F, phi2^T 3F -> F, [U^T | V^T] 2F -> F,
  // upd1^T F -> 2F, upd2^T 3F -> F
  DenseDev phi1T, phi2T, uvT, upd1T, upd2T;
};

struct PrecModel {      // the model cast and packed for one precision
  int prec = -1;
  void* emb = nullptr;  // [n_species][F] storage type
  // layer 0's phi of every species' embedding, [n_species][3F] storage type:
  // s before the first layer depends on the species alone, and phi acts on
  // each row by itself, so an atom's h of layer 0 is its species' row
  void* h0 = nullptr;
  std::vector<LayerDev> layers;
  std::vector<DenseDev> shared;                 // shared head layers
  std::vector<std::vector<DenseDev>> branch;    // [head][layer]
  void* head_table = nullptr;                   // device [head][layer][2] = (w, b)
  std::vector<DenseDev> blend;                  // branch-weighting MLP (empty: none)
  // reverse pass: transposed shared and branch layers (the branch's output
  // layer has none), device table [head][layer][2] = (w^T, null)
  bool has_T = false;
  std::vector<DenseDev> sharedT;
  std::vector<std::vector<DenseDev>> branchT;
  void* head_tableT = nullptr;
  std::vector<void*> allocs;
};

// ---- per-kernel event timing (painn_profile_*) ------------------------------
enum KernelClass {
  KC_GRAPH_PREP, KC_GRAPH_COUNT, KC_GRAPH_SCAN, KC_GRAPH_FILL, KC_EMBED, KC_PHI,
  KC_EDGE_PREP, KC_MESSAGE, KC_UPDATE, KC_HEADS, KC_ENERGY, KC_EXPORT,
  KC_TRANSPOSE, KC_BWD_HEADS, KC_BWD_UPDATE, KC_BWD_MESSAGE, KC_BWD_PHI, KC_FORCE,
  KC_TRAIN_REAL, KC_TRAIN_TANGENT, KC_TRAIN_ADAMW, KC_COUNT
};
struct Profiler;
// Record the start (begin = true) or end of a kernel of class `kc` on `s`;
// a no-op when `p` is null or disabled.
void prof_mark(Profiler* p, hipStream_t s, int kc, bool begin);

struct painn_ctx {
  int device = 0;
  Profiler* prof = nullptr;
  hipStream_t stream = nullptr;
  std::string err;
  DevStatus* h_status = nullptr;   // pinned host mirror of the graph status
  // forward workspace (grown on demand)
  void* ws = nullptr;
  size_t ws_bytes = 0;
  // reverse-pass workspace (saved activations and gradients; grown on demand)
  void* bws = nullptr;
  size_t bws_bytes = 0;
};

struct painn_model {
  painn_ctx* ctx = nullptr;
  Hyper hp;
  std::vector<double> master;      // FP64 weights in file order
  std::vector<size_t> offsets;     // offset of each array in `master`
  PrecModel* prec[3] = {nullptr, nullptr, nullptr};
};

struct painn_graph {
  painn_ctx* ctx = nullptr;
  int32_t B = 0, N = 0;
  long long E = 0;
  double cutoff = 0.0;
  int32_t species_min = 0, species_max = -1;
  bool any_pbc = false;
  // set only when the last build succeeded; a failed rebuild leaves buffers
  // half written, and every consumer of the graph refuses it until rebuilt
  bool valid = false;
  // device buffers (capacities in elements)
  int32_t* row_ptr = nullptr;  int32_t* counts = nullptr;
  int32_t* col = nullptr;      int32_t* shift = nullptr;
  int32_t* recv = nullptr;     // receiver of each edge (the CSR row, expanded)
  double* pos = nullptr;       int32_t* species = nullptr;
  int32_t* atom_struct = nullptr;
  double* cell = nullptr;      StructInfo* sinfo = nullptr;
  int32_t* struct_ptr = nullptr;
  long long* scan_tmp = nullptr;
  DevStatus* d_status = nullptr;
  // cell lists: per structure grid, per atom bin and wrap (fractional floor),
  // per bin count and start.  Structure b owns bins [2 lo_b + 27 b, ...) and
  // uses at most 2 n_b + 27 of them, so n_bins = 2 N + 27 B covers a batch.
  CellGrid* grid = nullptr;
  int32_t* bin_of = nullptr;   int32_t* wrap = nullptr;   int32_t* bin_atoms = nullptr;
  int32_t* bin_count = nullptr; int32_t* bin_start = nullptr;
  long long* bin_scan_tmp = nullptr;
  size_t n_bins = 0;
  // neighbour cap (0: none): the full CSR is built first, then each
  // receiver keeps its max_neighbors nearest edges in the public arrays above
  int32_t max_neighbors = 0;
  long long E_full = 0;
  int32_t* counts_cap = nullptr;  int32_t* row_ptr_full = nullptr;
  int32_t* col_full = nullptr;    int32_t* shift_full = nullptr;  int32_t* recv_full = nullptr;
  size_t cap_edges_full = 0, cap_atoms_cap = 0;
  size_t cap_atoms = 0, cap_struct = 0, cap_edges = 0, cap_scan = 0, cap_bins = 0, cap_bin_scan = 0;
  // edges grouped by sender (built on the first forces call, dropped by a
  // rebuild): t_edge[t_ptr[j] .. t_ptr[j+1]) are the ids of the edges whose
  // sender is j, ascending
  bool t_valid = false;
  int32_t* t_ptr = nullptr;    int32_t* t_edge = nullptr;   int32_t* t_count = nullptr;
  size_t cap_t_atoms = 0, cap_t_edges = 0;
};

// ---- kernel launchers (each enqueues on `s`, returns hipGetLastError) ------
hipError_t launch_graph_prep(hipStream_t s, Profiler* p, int B, int N, const int32_t* struct_ptr,
                             const double* pos, const int32_t* species, const double* cell,
                             const uint8_t* pbc, double cutoff, painn_graph* g);
hipError_t launch_graph_count(hipStream_t s, Profiler* p, painn_graph* g);
hipError_t launch_graph_scan(hipStream_t s, Profiler* p, painn_graph* g);
hipError_t launch_graph_fill(hipStream_t s, Profiler* p, painn_graph* g);
// neighbour cap: capped counts and their scan (before the readback), then
// the nearest-neighbour selection (after the full fill)
hipError_t launch_graph_cap_scan(hipStream_t s, Profiler* p, painn_graph* g);
hipError_t launch_graph_cap_select(hipStream_t s, Profiler* p, painn_graph* g);

struct ForwardArgs {
  const painn_model* m;
  const PrecModel* pm;
  const painn_graph* g;
  const int32_t* dataset_id;
  double* energies;
  // workspace
  void* s;      // [N][F] storage
  void* v[2];   // [N][3][F] storage, double buffered
  void* h;      // [N][3F] storage
  void* e;      // [N] accumulation type
  void* basis;           // [E + 16][kcols] storage type: radial basis rows
  void* einfo;           // [E][4] accumulation type: rhat, sender index
  void* head_plan;       // per-head counts and offsets (a few hundred bytes)
  void* head_tiles;      // [N H / 16 + 65] tiles of one head each (16 bytes)
  int32_t* head_order;   // [N H] (atom, head) entries grouped by head
  // blended heads (blend = true): composition [B][pad32(S)] (storage type),
  // head weights [B][H] and per-head atom energies [N][H] (accumulation type)
  bool blend;
  double skip;
  double* weights_out;   // [B][H] f64 or null
  void* comp;
  void* hw;
  void* eh;
  int stop_layer;          // run layers 0..stop_layer (forward: L-1)
  Profiler* prof;
  double* s_out;           // feature export (may be null)
  double* v_out;
  void* save;              // per-layer activations for the reverse pass (may be null)
  // (FP64) the message kernel's LDS image of each layer's filter, written per
  // layer before the message (MSG64_IMAGE_BYTES; may be null: the kernel
  // then gathers its filter fragments itself)
  void* msg_img;
};

// Upper bound of that image: 2-way channel split x 4 groups x (6 x 4 fragment
// pairs x 64 lanes + 3 x 16 bias pairs) x 16 bytes, at F <= 384 at most 12
// groups in all.
constexpr size_t MSG64_IMAGE_BYTES = (size_t)12 * (6 * 4 * 64 + 3 * 16) * 16;

// The activations a forward run keeps for the reverse pass (storage type,
// element size es).  Layer l: S(l) = s before the message [N][F], V(l) = v
// [N][3F], H(l) = phi(s) [N][3F], Smid(l), Vmid(l) = s and v after the
// message; S(L), V(L) = the final s and v.  Then per layer the update's
// intermediates: UV(l) = [U v[c] | V v[c]] for c = x, y, z [N][3][2F], Z(l) =
// the gate MLP's pre-activation [N][F], Agate(l) = [a_vv | a_sv] [N][2F].
struct SaveLayout {
  char* base;
  size_t N, F, es;
  int L;
  __host__ __device__ SaveLayout(void* b, size_t n, size_t f, int l, size_t e)
      : base((char*)b), N(n), F(f), es(e), L(l) {}
  __host__ __device__ void* UV(int l) const { return base + ((size_t)L * 11 + 4 + (size_t)l * 9) * N * F * es; }
  __host__ __device__ void* Z(int l) const { return (char*)UV(l) + 6 * N * F * es; }
  __host__ __device__ void* Agate(int l) const { return (char*)Z(l) + N * F * es; }
  __host__ __device__ void* S(int l) const { return base + (size_t)l * 11 * N * F * es; }
  __host__ __device__ void* V(int l) const { return (char*)S(l) + N * F * es; }
  __host__ __device__ void* H(int l) const { return (char*)V(l) + 3 * N * F * es; }
  __host__ __device__ void* Smid(int l) const { return (char*)H(l) + 3 * N * F * es; }
  __host__ __device__ void* Vmid(int l) const { return (char*)Smid(l) + N * F * es; }
  static size_t bytes(size_t N, size_t F, int L, size_t es) { return ((size_t)L * 20 + 4) * N * F * es; }
};

// Atoms grouped by head (the heads kernels' counting sort): per-head counts
// and offsets, then tiles of atoms of one head.
constexpr int HEADS_MAX = 64;
struct HeadPlan {
  int32_t count[HEADS_MAX];   // valid atoms per head
  int32_t start[HEADS_MAX];   // first slot of the head in the atom order
  int32_t cursor[HEADS_MAX];  // scatter cursor
  int32_t n_tiles;
};
struct HeadTile {
  int32_t head, begin, end, pad;   // slots [begin, end) of the atom order
};

// Reverse pass (FP64 / FP32): forces -dE/dx from a forward run with a save
// area.  Gradient buffers hold the accumulation type.
struct BackwardArgs {
  const painn_model* m;
  const PrecModel* pm;
  const painn_graph* g;
  const int32_t* dataset_id;
  void* save;               // the forward's save area
  const void* einfo;        // [E][4] the forward's edge info: rhat in 0..2
  // in the order of the sender-grouped edge list (E + 16 rows): the basis
  // rows, their derivatives d/dd, and (rhat, receiver index)
  void* basis_t;
  void* dbasis;
  void* einfo_t;
  const void* head_plan;    // the forward's grouping of atoms by head
  const void* head_tiles;
  const int32_t* head_order;
  void* gs;  void* gv;      // dE/ds [N][F], dE/dv [N][3F] at a layer boundary
  void* gs2; void* gv2;     // the same after a layer's message
  void* gh;                 // dE/dh [N][3F]
  void* scratch;            // per-atom intermediates [N][scratch_w]
  int scratch_w;
  void* xbuf;               // operand buffers in global memory for tiles too wide for the LDS
  size_t xbuf_bytes;
  void* eg;                 // [E][NW][4] per-edge partials dE/dd, dE/drhat
  double* gr;               // [E][3] dE/dr per edge
  double* forces;           // [N][3] output
  // blended heads: the forward's head weights [B][H] (accumulation type),
  // the skip threshold, and per-(atom, head) dE/ds slots [N][H][F]
  bool blend;
  double skip;
  const void* hw;
  void* g_heads;
  Profiler* prof;
};
hipError_t launch_backward(hipStream_t s, int prec, BackwardArgs& a);
// The fixed scratch of painn_forward_noalloc: its size, the once-per-device
// lookup of its address (painn_create calls it with the device current) and
// that address (null before a successful lookup).
constexpr size_t NOALLOC_SCRATCH_BYTES = (size_t)64 << 20;
hipError_t noalloc_scratch_init(int device);
void* noalloc_scratch(int device);
// workgroups of the reverse heads kernel (a persistent grid; each has its
// own 16 scratch rows and, for wide layers, its own operand buffers)
constexpr int HB_GRID = 2048;
// the sender-grouped edge list of a graph
hipError_t launch_transpose(hipStream_t s, Profiler* p, painn_graph* g);
size_t forward_workspace_bytes(int prec, int N, long long E, int F, int kcols, int B, int H,
                               int S, bool blend);
hipError_t launch_forward(hipStream_t s, int prec, ForwardArgs& a);
// pm->h0 from pm->emb and layer 0's phi (enqueued on s; out holds
// n_species x 3F storage elements)
hipError_t launch_phi0_table(hipStream_t s, int prec, int F, int n_species, const PrecModel* pm, void* out);
