/*
 * painn.h - C ABI of the MI355X (gfx950) batched PaiNN screening forward pass.
 *
 * The operation is the one the paper runs over 1.1 billion structures
 * (section "Inference on Billions of Atomistic Structures on Frontier"): for a
 * batch of many small molecules and periodic cells, build the radius graph
 * (lead model: cutoff radius, Table 5), run the PaiNN interaction layers
 * (PaiNN is the lead backbone chosen in section "Flagship Training of Top HPO
 * Models"; message and update blocks as published by Schuett et al. 2021),
 * and read out one energy per structure through per-dataset heads (Table 5:
 * shared layers + branch layers, 16 graph-level branches; section "Multi-task
 * learning for imbalanced, heterogeneous multi-fidelity data").  Precision is
 * a per-call choice among FP64, FP32 and BF16 (section "Precision-sensitivity
 * characterization at inference and fine-tuning stage").
 *
 * Conventions for every entry point:
 *  - Return value: PAINN_OK (0) or a negative painn_status.  Nothing throws or
 *    aborts; after an error, painn_last_error(ctx) describes it.
 *  - Array arguments are DEVICE pointers (memory of the context's device),
 *    owned by the caller, unless a comment says "host".  They are read in the
 *    order of the context's stream; the caller keeps them alive and unchanged
 *    until that stream has passed the call.
 *  - Opaque objects (context, model, graph) are owned by the library and are
 *    released only by the matching *_free / painn_destroy.
 *  - All work is enqueued on the context's HIP stream.  The only host
 *    synchronisation is inside painn_build_graph (it reads back the edge
 *    count) and painn_synchronize.
 *  - A context is not thread-safe; use one context per host thread.
 */
#ifndef PAINN_H
#define PAINN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PAINN_OK = 0,
  PAINN_E_ARG = -1,          /* invalid argument (null pointer, size, cutoff, struct_ptr) */
  PAINN_E_OOM = -2,          /* device or host allocation failed */
  PAINN_E_HIP = -3,          /* a HIP runtime call failed */
  PAINN_E_FILE = -4,         /* weight file cannot be opened or read */
  PAINN_E_FORMAT = -5,       /* weight file malformed (magic, header, size) */
  PAINN_E_SPECIES = -6,      /* a species index is outside [0, n_species) */
  PAINN_E_COINCIDENT = -7,   /* two atoms (or an atom and a periodic image) at distance 0 */
  PAINN_E_UNSUPPORTED = -8   /* shape or option the kernels do not implement */
} painn_status;

typedef enum {
  PAINN_FP64 = 0,            /* weights, features and accumulation in FP64 */
  PAINN_FP32 = 1,            /* weights, features and accumulation in FP32 */
  PAINN_BF16 = 2             /* BF16 weights and stored features, FP32 accumulation */
} painn_precision;

typedef struct painn_ctx painn_ctx;
typedef struct painn_model painn_model;
typedef struct painn_graph painn_graph;

/* ---- context ---------------------------------------------------------- */

/* Create a context on HIP device `device`, enqueueing on `hip_stream` (a
 * hipStream_t; NULL = the device's null stream).  The library does not take
 * ownership of the stream.  *out receives the context. */
painn_status painn_create(int device, void* hip_stream, painn_ctx** out);
/* Change the stream of an existing context (same device). */
painn_status painn_set_stream(painn_ctx* ctx, void* hip_stream);
/* Release the context and its workspace.  Models and graphs created on it
 * must be freed first.  NULL is accepted. */
painn_status painn_destroy(painn_ctx* ctx);
/* Message of the last error on this context (never NULL; "" after success). */
const char* painn_last_error(const painn_ctx* ctx);
/* Static name of a status code. */
const char* painn_status_string(int status);
/* Block the host until all work enqueued by the context has finished. */
painn_status painn_synchronize(painn_ctx* ctx);

/* ---- model -------------------------------------------------------------- */

/* Load an FP64 weight file (host path).  Format, little-endian:
 *   char magic[8] = "PAINNW01";
 *   int32 F, K, L, n_species, n_heads, rbf_type, n_shared, n_branch;
 *     rbf_type 0: Gaussians exp(-gamma (d - mu_k)^2), mu_k = k r_c / (K - 1),
 *     gamma = 1 / (2 Delta^2), Delta = r_c / (K - 1); 1: Bessel sin(n pi d / r_c) / d,
 *     n = 1..K (the lead model's basis, Table 5); both under the cosine cutoff;
 *   float64 cutoff;
 *   int32 shared_dims[n_shared];   output width of each shared head layer
 *   int32 branch_dims[n_branch];   output width of each branch layer (last = 1)
 *   zero padding to a multiple of 8 bytes;
 *   float64 arrays, row-major, dense weights stored [out, in]:
 *     emb[n_species, F];
 *     per layer: phi_w1[F,F] phi_b1[F] phi_w2[3F,F] phi_b2[3F]
 *                filt_w[3F,K] filt_b[3F] U[F,F] V[F,F]
 *                upd_w1[F,2F] upd_b1[F] upd_w2[3F,F] upd_b2[3F];
 *     per shared layer m: w[shared_dims[m], in] b[shared_dims[m]];
 *     per head h, per branch layer m: w[branch_dims[m], in] b[branch_dims[m]].
 *   optional, the branch-weighting MLP (section "Composition-conditioned branch
 *   weighting"): char magic[8] = "BLENDW01"; int32 n_hidden;
 *   int32 hidden_dims[n_hidden]; zero padding to a multiple of 8 bytes;
 *   float64 layers w[out, in] b[out] from n_species through the hidden widths
 *   to n_heads.
 *   optional, a neighbour cap: char magic[8] = "NBRCAP01"; int32 max_neighbors;
 *   int32 0.  Optional sections follow the arrays, each at most once, in any
 *   order.
 * The split of phi's output is [s | v | rhat] and of the update MLP's output
 * [a_vv | a_sv | a_ss].  Supported: 1 <= F <= 384 (the kernels run at
 * F = 64, 128, 256 or 384; any other width is zero-padded on load to the next
 * of them, which leaves every energy unchanged), 2 <= K <= 64, 1 <= L <= 16,
 * 1 <= n_heads <= 64, head widths in [1, 1024], branch_dims[last] = 1; with
 * the branch-weighting MLP n_species <= 256 and widths <= 1024.
 * Errors: PAINN_E_ARG (null argument), PAINN_E_FILE (the path cannot be
 * opened or read), PAINN_E_FORMAT (bad magic, truncated or oversized
 * arrays, trailing bytes, a malformed or repeated optional section, a
 * non-finite weight), PAINN_E_UNSUPPORTED (a shape outside the ranges
 * above), PAINN_E_OOM. */
painn_status painn_model_load(painn_ctx* ctx, const char* path, painn_model** out);
/* Same, from a host buffer holding the file's bytes (copied; the buffer may
 * be released after the call). */
painn_status painn_model_load_buffer(painn_ctx* ctx, const void* data, size_t nbytes,
                                     painn_model** out);
/* Hyperparameters of a model (host outputs; any pointer may be NULL). */
painn_status painn_model_info(const painn_model* model, int32_t* F, int32_t* K, int32_t* L,
                              int32_t* n_species, int32_t* n_heads, double* cutoff);
/* Optional parts of a model (host outputs; either pointer may be NULL):
 * *has_blend = 1 when it carries a branch-weighting MLP, else 0;
 * *max_neighbors = its neighbour cap (0: none). */
painn_status painn_model_options(const painn_model* model, int32_t* has_blend, int32_t* max_neighbors);
painn_status painn_model_free(painn_model* model);

/* ---- graph -------------------------------------------------------------- */

/* Build the radius graph of a batch of B structures with N atoms in total.
 * Edges are all (i <- j, n) with i, j in the same structure, n an integer
 * image vector (n_k = 0 on non-periodic axes), (i, j, n) != (i, i, 0), and
 *   t = (n0*a + n1*b) + n2*c,  r = (x_j - x_i) + t,
 *   d2 = (r.x*r.x + r.y*r.y) + r.z*r.z  <  cutoff*cutoff
 * evaluated in IEEE FP64 in exactly this order without fused multiply-add, so
 * the edge set is bit-exact.  Every periodic image within the cutoff is kept.
 * The CSR is sorted by receiver i, then sender j, then (n0, n1, n2).
 *   struct_ptr [B+1] int32: atoms of structure b are [struct_ptr[b], struct_ptr[b+1]);
 *                           struct_ptr[0] = 0, non-decreasing, struct_ptr[B] = N.
 *   pos        [N,3] float64, Angstrom.
 *   species    [N]   int32, checked against the model at painn_forward.
 *   cell       [B,3,3] float64, rows are the lattice vectors a, b, c; may be
 *              NULL when pbc is NULL.
 *   pbc        [B,3] uint8, nonzero = periodic along that lattice vector; NULL
 *              = no periodic axis anywhere.  A periodic cell must be non-singular.
 * The graph copies what it needs (positions, species, cells), so the inputs
 * may change after the call's stream position.  If *inout is NULL a new graph
 * is created; otherwise *inout is rebuilt in place, reusing its memory.  When
 * an in-place rebuild fails after its arguments passed the host checks, the
 * graph is left unusable: painn_graph_csr, painn_forward* and painn_forces*
 * return PAINN_E_ARG for it until a later build succeeds (it may still be
 * rebuilt or freed).  Synchronises the stream once.  Errors: PAINN_E_ARG (bad sizes, cutoff not
 * finite and > 0, malformed struct_ptr, singular periodic cell, more than
 * 2^31-1 edges, image range beyond +-127), PAINN_E_COINCIDENT. */
painn_status painn_build_graph(painn_ctx* ctx, int32_t n_struct, int32_t n_atoms,
                               const int32_t* struct_ptr, const double* pos,
                               const int32_t* species, const double* cell,
                               const uint8_t* pbc, double cutoff, painn_graph** inout);
/* Same, keeping at most max_neighbors edges per receiver (0: every edge): the
 * nearest ones, by the exact d2 above, ties to the lower sender and then the
 * lower shift (n0, n1, n2); the kept edges stay in (sender, shift) order.
 * The lead model keeps 20 (Table 5).  A model whose weight file carries a
 * neighbour cap runs only on a graph built with that cap. */
painn_status painn_build_graph_capped(painn_ctx* ctx, int32_t n_struct, int32_t n_atoms,
                                      const int32_t* struct_ptr, const double* pos,
                                      const int32_t* species, const double* cell,
                                      const uint8_t* pbc, double cutoff, int32_t max_neighbors,
                                      painn_graph** inout);
/* Borrow the CSR of a graph (device pointers valid until the graph is rebuilt
 * or freed): row_ptr [N+1] int32, col [E] int32 (batch-global sender index),
 * shift [E] int32 packing (n0, n1, n2) as signed bytes 0, 1, 2 (byte 3 = 0).
 * Host outputs; any may be NULL. */
painn_status painn_graph_csr(const painn_graph* graph, int64_t* n_edges, int32_t* n_atoms,
                             int32_t* n_struct, const int32_t** row_ptr, const int32_t** col,
                             const int32_t** shift);
painn_status painn_graph_free(painn_graph* graph);

/* ---- forward ------------------------------------------------------------ */

/* Per-structure energies E_b = sum over atoms i of structure b of e_i, where
 * e_i is the head of the structure's dataset applied to atom i's final
 * scalar features.
 *   dataset_id [B] int32 in [0, n_heads), or NULL = head 0 for every structure.
 *   energies   [B] float64 output, written on the stream.
 * The graph must have been built with the model's cutoff.  Errors:
 * PAINN_E_ARG (cutoff mismatch, null pointers), PAINN_E_SPECIES,
 * PAINN_E_UNSUPPORTED.  Asynchronous, so a dataset id outside [0, n_heads)
 * cannot be reported as a status: that structure's energy is written as NaN. */
painn_status painn_forward(painn_ctx* ctx, const painn_model* model, const painn_graph* graph,
                           const int32_t* dataset_id, painn_precision precision,
                           double* energies);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * energies as painn_forward, computed by the same kernels, with the forward's
 * workspace carved from one fixed device array of 64 MiB
 * (NOALLOC_SCRATCH_BYTES) that the library holds on each device from its
 * first use until the process ends.  The call allocates nothing: the model
 * must already hold its packed weights for this precision (run painn_forward
 * once at this precision first; otherwise PAINN_E_ARG), the graph is built
 * beforehand, and per-kernel event timing (painn_profile_enable) is not
 * recorded for it.  A batch whose workspace exceeds 64 MiB (about 9,000
 * atoms at F = 128 in FP32; fewer at wider F, more in BF16) is refused with
 * PAINN_E_ARG, naming the bytes it needs.  Every call on a device shares that
 * device's array: calls that overlap in time on one device (on different
 * streams or contexts) race and must be ordered by the caller.  Arguments and
 * other errors as painn_forward. */
painn_status painn_forward_noalloc(painn_ctx* ctx, const painn_model* model, const painn_graph* graph,
                                   const int32_t* dataset_id, painn_precision precision,
                                   double* energies);

/* Per-structure energies with every head blended (sections
 * "Composition-conditioned branch weighting" and "Optimizing the Inference
 * Pipeline", branch skipping): the encoder runs once; structure b's
 * composition vector (fraction of its atoms of each species) goes through the
 * model's branch-weighting MLP to softmax weights w_bh over the heads, and
 * E_b = sum over heads h with w_bh >= skip_threshold of w_bh E_bh, where E_bh
 * is head h's energy of structure b.  skip_threshold = 0 keeps every head;
 * skipped heads are not computed and the kept weights are not renormalised.
 *   energies [B] float64 output; weights [B, n_heads] float64 output of the
 *   weights w_bh, or NULL.  Both written on the stream.
 * Errors: as painn_forward; PAINN_E_UNSUPPORTED when the model has no
 * branch-weighting MLP; PAINN_E_ARG for a negative or non-finite threshold. */
painn_status painn_forward_blend(painn_ctx* ctx, const painn_model* model, const painn_graph* graph,
                                 painn_precision precision, double skip_threshold, double* energies,
                                 double* weights);

/* Energies and forces (the paper's screening throughput counts both, and its
 * largest single inference gain computes the force gradient in the same pass
 * as the energy: section "Optimizing the Inference Pipeline", Fig. 4).
 * Forces are F_i = -dE/dx_i with E the total energy of atom i's structure,
 * by a hand-written reverse pass through the heads, every layer's update,
 * message and phi, the radial filter and the edge geometry.  The graph is
 * held fixed: the cosine cutoff makes every message vanish with zero slope
 * at r_c, and the neighbour cap is piecewise constant in the positions.
 *   dataset_id [B] as in painn_forward (NULL = head 0).
 *   energies   [B] float64 output (the same values as painn_forward).
 *   forces     [N, 3] float64 output (eV/Angstrom for energies in eV).
 * Both written on the stream; the reverse pass keeps every layer's
 * activations (about (20 L + 4) N F values of the precision's storage type
 * plus per-edge buffers) in a context workspace grown on demand.  The first
 * call on a graph also groups its edges by sender (kept until the graph is
 * rebuilt).  As in painn_forward, a structure whose dataset id is outside
 * [0, n_heads) gets NaN energy, and here NaN forces on its atoms.  Errors: as
 * painn_forward; PAINN_E_UNSUPPORTED for BF16. */
painn_status painn_forces(painn_ctx* ctx, const painn_model* model, const painn_graph* graph,
                          const int32_t* dataset_id, painn_precision precision, double* energies,
                          double* forces);

/* Energies and forces with every head blended (as painn_forward_blend): the
 * head weights w_bh depend on the composition only, so the forces are
 * -sum over kept heads of w_bh dE_bh/dx.  Arguments and errors as
 * painn_forward_blend and painn_forces (weights may be NULL). */
painn_status painn_forces_blend(painn_ctx* ctx, const painn_model* model, const painn_graph* graph,
                                painn_precision precision, double skip_threshold, double* energies,
                                double* forces, double* weights);

/* Test hook: run layers 0..layer (layer = -1: embedding only) and write the
 * scalar features s [N,F] and vector features v [N,3,F] (float64) reached
 * there.  Same arguments and errors as painn_forward. */
painn_status painn_forward_features(painn_ctx* ctx, const painn_model* model,
                                    const painn_graph* graph, painn_precision precision,
                                    int32_t layer, double* s_out, double* v_out);

/* ---- training ----------------------------------------------------------- */

/* One FP64 training step on energies and forces (section "Flagship Training
 * of Top HPO Models"; Table "Lead PaiNN model configuration": MAE loss, force
 * weight ~94.8, AdamW at learning rate 6.34e-4, FP64).  The loss over a batch
 * of B structures and N atoms is
 *   L = (1/B) sum_b |E_b - E*_b| + force_weight (1/(3N)) sum_{i,c} |F_ic - F*_ic|
 * with F = -dE/dx (forces as painn_forces, dataset-id heads).  A step runs the
 * forward and the reverse pass to the forces, then the gradient of L with
 * respect to every weight (the force term through the derivative of the
 * weight gradient along the force residuals' signs), then one AdamW update
 * (decoupled weight decay, bias-corrected moments) of every weight.  The
 * trainer keeps its own FP64 copy of the weights (at the model's own width,
 * in the weight file's order) and the optimizer state; the model it was made
 * from is not changed. */
typedef struct painn_trainer painn_trainer;
typedef struct {
  double lr;            /* learning rate (6.34e-4) */
  double beta1, beta2;  /* AdamW moment decays (0.9, 0.999) */
  double eps;           /* AdamW denominator offset (1e-8) */
  double weight_decay;  /* decoupled weight decay (0.01) */
  double force_weight;  /* the loss's force weight (94.8) */
} painn_train_config;

/* Create a trainer from a model's weights.  cfg is a host pointer (NULL: the
 * values in parentheses above).  Errors: PAINN_E_ARG (null model, values out
 * of range: lr, eps, weight_decay, force_weight finite and >= 0 (eps > 0),
 * 0 <= beta < 1), PAINN_E_OOM. */
painn_status painn_trainer_create(painn_ctx* ctx, const painn_model* model, const painn_train_config* cfg,
                                  painn_trainer** out);
/* One step on a batch: the graph (built with the model's cutoff and
 * neighbour cap from the batch's positions), dataset_id [B] (device; NULL =
 * head 0), reference energies energy_ref [B] and forces force_ref [N, 3]
 * (device, float64).  loss [3] (device float64, or NULL) receives L, the
 * energy MAE and the force MAE at the weights before the update.  A dataset
 * id outside [0, n_heads) makes the loss NaN (asynchronous: not a status).
 * Errors: PAINN_E_ARG (null or mismatched graph, null references),
 * PAINN_E_SPECIES, PAINN_E_UNSUPPORTED (more than 2^31 - 1 edges or 3 N F
 * values), PAINN_E_OOM, PAINN_E_HIP.  Deterministic: every reduction runs in
 * a fixed order. */
painn_status painn_trainer_step(painn_trainer* tr, const painn_graph* graph, const int32_t* dataset_id,
                                const double* energy_ref, const double* force_ref, double* loss);
/* The number of weights (host), and copies (device, float64 [n_params], in
 * the weight file's array order at the model's own width; either may be
 * NULL) of the current weights and of the last step's gradient. */
painn_status painn_trainer_params(const painn_trainer* tr, int64_t* n_params, double* params, double* grad);
painn_status painn_trainer_free(painn_trainer* tr);

/* ---- tracing ------------------------------------------------------------ */

/* Per-kernel timing with HIP events on the context's stream (the build's
 * counterpart of the paper's application timers, section "How Performance
 * Was Measured").  While enabled, every kernel launch is bracketed by two
 * event records on the stream; nothing synchronises until painn_profile_read.
 * enable = 0 stops recording (accumulated results are kept). */
painn_status painn_profile_enable(painn_ctx* ctx, int enable);
/* Synchronise the stream, then write per kernel class (at most n_max): its
 * name (static string), accumulated GPU milliseconds and launch count since
 * the last read; reset the accumulators.  names, ms, launches are host arrays
 * of n_max entries; *n_out receives the number of classes written. */
painn_status painn_profile_read(painn_ctx* ctx, int32_t n_max, const char** names, double* ms,
                                int64_t* launches, int32_t* n_out);

#ifdef __cplusplus
}
#endif
#endif /* PAINN_H */
