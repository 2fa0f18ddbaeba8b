// Host-only reader of the FP64 weight file (format in painn.h, at
// painn_model_load).  No HIP: this translation unit is also built on its own,
// with the host sanitizers, by the CPU tests.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "painn.h"

struct Hyper {
  int F = 0;          // feature width the kernels run at (64, 128, 256, 384)
  int F_logical = 0;  // the model's own width (<= F; the rest is zero padding)
  int K = 0, L = 0, n_species = 0, n_heads = 0, rbf_type = 0;
  double cutoff = 0.0;
  std::vector<int> shared_dims, branch_dims;
  std::vector<int> blend_dims;   // hidden widths of the branch-weighting MLP
  bool has_blend = false;
  int max_neighbors = 0;         // neighbour cap the model was trained with (0: none)
};

// Names of the per-layer arrays in file order.
enum { A_PHI_W1, A_PHI_B1, A_PHI_W2, A_PHI_B2, A_FILT_W, A_FILT_B, A_U, A_V,
       A_UPD_W1, A_UPD_B1, A_UPD_W2, A_UPD_B2, A_PER_LAYER };

struct WeightFile {
  Hyper hp;
  std::vector<double> master;    // every array in file order, FP64
  std::vector<size_t> offsets;   // start of each array in `master`
};

// Parse n bytes of a weight file.  On success returns PAINN_OK and fills
// *out, with the feature width padded to the next width the kernels run at
// (hp.F_logical keeps the file's F).  On failure returns PAINN_E_FORMAT,
// PAINN_E_UNSUPPORTED or PAINN_E_OOM, sets *err and leaves *out unspecified.
// Reads no byte outside [buf, buf + n).
int parse_weight_file(const unsigned char* buf, size_t n, WeightFile* out, std::string* err);
