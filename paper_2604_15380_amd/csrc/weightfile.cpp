// Host-only reader of the FP64 weight file: header checks, array sizes,
// optional sections, and the zero padding of the feature width.  Every read
// is bounds-checked against the buffer length.
#include "weightfile.h"

#include <string.h>

#include <cmath>
#include <new>

// The kernels run at feature widths 64, 128, 256 and 384.  A model of any
// other width F <= 384 is padded with zeros to the next of them: padded
// channels of s, v and h stay exactly 0 (zero embedding columns, zero rows
// and biases of every layer producing them) and never reach a real channel
// (zero columns of every layer reading them), so the energies are those of
// the F-wide model.  Every array of the master copy is re-laid out at the
// padded width; dimensions made of P blocks of F channels ([h_s | h_v | h_r],
// [s ; |Vv|], [a_vv | a_sv | a_ss]) are padded block by block.
static int padded_width(int F) { return F <= 64 ? 64 : F <= 128 ? 128 : F <= 256 ? 256 : 384; }

static void pad_feature_width(WeightFile* m) {
  Hyper& hp = m->hp;
  const int F = hp.F, Fp = padded_width(F);
  if (Fp == F) return;
  // (rows, cols) of each array in file order; a dimension given as -P means
  // P blocks of F channels
  struct Dim { int rows, cols; };
  std::vector<Dim> dims;
  dims.push_back({hp.n_species, -1});
  for (int l = 0; l < hp.L; ++l) {
    const Dim per[A_PER_LAYER] = {{-1, -1}, {-1, 1}, {-3, -1}, {-3, 1}, {-3, hp.K}, {-3, 1},
                                  {-1, -1}, {-1, -1}, {-1, -2}, {-1, 1}, {-3, -1}, {-3, 1}};
    for (const Dim& d : per) dims.push_back(d);
  }
  int din = -1;
  for (int d : hp.shared_dims) { dims.push_back({d, din}); dims.push_back({d, 1}); din = d; }
  for (int h = 0; h < hp.n_heads; ++h) {
    int di = din;
    for (int d : hp.branch_dims) { dims.push_back({d, di}); dims.push_back({d, 1}); di = d; }
  }
  const size_t n_main = dims.size();
  auto ext = [&](int d, int w) { return d < 0 ? (size_t)(-d) * w : (size_t)d; };
  auto map = [&](int d, size_t x) { return d < 0 ? (x / F) * Fp + x % F : x; };
  std::vector<double> out;
  std::vector<size_t> offs;
  for (size_t a = 0; a < m->offsets.size(); ++a) {
    const double* src = m->master.data() + m->offsets[a];
    offs.push_back(out.size());
    if (a >= n_main) {                       // branch-weighting MLP: unchanged
      const size_t n = (a + 1 < m->offsets.size() ? m->offsets[a + 1] : m->master.size()) - m->offsets[a];
      out.insert(out.end(), src, src + n);
      continue;
    }
    const Dim d = dims[a];
    const size_t R = ext(d.rows, F), C = ext(d.cols, F), Rp = ext(d.rows, Fp), Cp = ext(d.cols, Fp);
    const size_t o = out.size();
    out.resize(o + Rp * Cp, 0.0);
    for (size_t r = 0; r < R; ++r)
      for (size_t c = 0; c < C; ++c) out[o + map(d.rows, r) * Cp + map(d.cols, c)] = src[r * C + c];
  }
  m->master.swap(out);
  m->offsets.swap(offs);
  hp.F = Fp;
}

int parse_weight_file(const unsigned char* buf, size_t n, WeightFile* out, std::string* err) {
  auto fail = [&](int st, const char* msg) {
    *err = msg;
    return st;
  };
  if (n < 48 || memcmp(buf, "PAINNW01", 8) != 0)
    return fail(PAINN_E_FORMAT, "weight file: bad magic or truncated header");
  int32_t h[8];
  memcpy(h, buf + 8, sizeof(h));
  Hyper hp;
  hp.F = h[0]; hp.K = h[1]; hp.L = h[2]; hp.n_species = h[3]; hp.n_heads = h[4];
  hp.rbf_type = h[5];
  const int ns = h[6], nb = h[7];
  memcpy(&hp.cutoff, buf + 40, 8);
  if (ns < 0 || ns > 16 || nb < 1 || nb > 16)
    return fail(PAINN_E_FORMAT, "weight file: bad head layer counts");
  size_t off = 48;
  if (n < off + 4 * (size_t)(ns + nb)) return fail(PAINN_E_FORMAT, "weight file: truncated");
  for (int i = 0; i < ns; ++i) { int32_t d; memcpy(&d, buf + off, 4); off += 4; hp.shared_dims.push_back(d); }
  for (int i = 0; i < nb; ++i) { int32_t d; memcpy(&d, buf + off, 4); off += 4; hp.branch_dims.push_back(d); }
  off += (8 - off % 8) % 8;
  if (hp.F < 1 || hp.F > 384) return fail(PAINN_E_UNSUPPORTED, "F must be in [1, 384]");
  if (hp.K < 2 || hp.K > 64) return fail(PAINN_E_UNSUPPORTED, "K must be in [2, 64]");
  if (hp.L < 1 || hp.L > 16) return fail(PAINN_E_UNSUPPORTED, "L must be in [1, 16]");
  if (hp.n_species < 1 || hp.n_species > 1024) return fail(PAINN_E_FORMAT, "bad n_species");
  if (hp.n_heads < 1 || hp.n_heads > 64) return fail(PAINN_E_UNSUPPORTED, "n_heads must be in [1, 64]");
  if (hp.rbf_type != 0 && hp.rbf_type != 1)
    return fail(PAINN_E_UNSUPPORTED, "radial basis must be 0 (Gaussian) or 1 (Bessel)");
  if (!(hp.cutoff > 0.0) || !std::isfinite(hp.cutoff)) return fail(PAINN_E_FORMAT, "bad cutoff");
  for (int d : hp.shared_dims)
    if (d < 1 || d > 1024) return fail(PAINN_E_UNSUPPORTED, "head widths must be in [1, 1024]");
  for (int d : hp.branch_dims)
    if (d < 1 || d > 1024) return fail(PAINN_E_UNSUPPORTED, "head widths must be in [1, 1024]");
  if (hp.branch_dims.back() != 1) return fail(PAINN_E_FORMAT, "last branch layer must have width 1");
  // array sizes in file order
  std::vector<size_t> sizes;
  const size_t F = hp.F, K = hp.K;
  sizes.push_back(hp.n_species * F);
  for (int l = 0; l < hp.L; ++l) {
    size_t per[A_PER_LAYER] = {F * F, F, 3 * F * F, 3 * F, 3 * F * K, 3 * F, F * F, F * F,
                               2 * F * F, F, 3 * F * F, 3 * F};
    for (size_t s : per) sizes.push_back(s);
  }
  size_t din = F;
  for (int d : hp.shared_dims) { sizes.push_back((size_t)d * din); sizes.push_back(d); din = d; }
  for (int hh = 0; hh < hp.n_heads; ++hh) {
    size_t di = din;
    for (int d : hp.branch_dims) { sizes.push_back((size_t)d * di); sizes.push_back(d); di = d; }
  }
  size_t total = 0;
  for (size_t s : sizes) total += s;
  const size_t main_total = total;
  // optional sections after the main arrays, each at most once, any order:
  //   'BLENDW01', int32 n_hidden, the hidden widths, zero padding to 8 bytes,
  //     then the branch-weighting MLP's layers (composition [n_species] ->
  //     hidden ... -> n_heads), each [out, in] + bias;
  //   'NBRCAP01', int32 max_neighbors, int32 0.
  size_t blend_off = 0;
  size_t bo = off + 8 * main_total;
  bool has_cap = false;
  while (bo < n) {
    if (n < bo + 16) return fail(PAINN_E_FORMAT, "weight file: size does not match its header");
    if (memcmp(buf + bo, "BLENDW01", 8) == 0 && !hp.has_blend) {
      int32_t nh;
      memcpy(&nh, buf + bo + 8, 4);
      if (nh < 0 || nh > 8 || n < bo + 12 + 4 * (size_t)nh)
        return fail(PAINN_E_FORMAT, "weight file: bad branch-weighting section");
      bo += 12;
      for (int i = 0; i < nh; ++i) { int32_t d; memcpy(&d, buf + bo, 4); bo += 4; hp.blend_dims.push_back(d); }
      bo += (8 - bo % 8) % 8;
      for (int d : hp.blend_dims)
        if (d < 1 || d > 1024) return fail(PAINN_E_UNSUPPORTED, "branch-weighting widths must be in [1, 1024]");
      if (hp.n_species > 256) return fail(PAINN_E_UNSUPPORTED, "branch weighting needs n_species <= 256");
      size_t di = hp.n_species, cnt = 0;
      std::vector<int> dims = hp.blend_dims;
      dims.push_back(hp.n_heads);
      for (int d : dims) {
        sizes.push_back((size_t)d * di);
        sizes.push_back(d);
        cnt += (size_t)d * di + d;
        di = d;
      }
      if (n < bo + 8 * cnt)
        return fail(PAINN_E_FORMAT, "weight file: branch-weighting section is truncated");
      total += cnt;
      hp.has_blend = true;
      blend_off = bo;
      bo += 8 * cnt;
    } else if (memcmp(buf + bo, "NBRCAP01", 8) == 0 && !has_cap) {
      int32_t c;
      memcpy(&c, buf + bo + 8, 4);
      if (c < 1) return fail(PAINN_E_FORMAT, "weight file: neighbour cap must be >= 1");
      hp.max_neighbors = c;
      has_cap = true;
      bo += 16;
    } else {
      return fail(PAINN_E_FORMAT, "weight file: size does not match its header");
    }
  }
  if (bo != n) return fail(PAINN_E_FORMAT, "weight file: size does not match its header");
  WeightFile* m = out;
  m->hp = hp;
  m->offsets.clear();
  try {
    m->master.resize(total);
  } catch (const std::bad_alloc&) {
    return fail(PAINN_E_OOM, "host allocation failed");
  }
  memcpy(m->master.data(), buf + off, 8 * main_total);
  if (hp.has_blend) memcpy(m->master.data() + main_total, buf + blend_off, 8 * (total - main_total));
  size_t o = 0;
  for (size_t s : sizes) { m->offsets.push_back(o); o += s; }
  for (double x : m->master)
    if (!std::isfinite(x)) return fail(PAINN_E_FORMAT, "weight file: non-finite weight");
  m->hp.F_logical = hp.F;
  pad_feature_width(m);
  return PAINN_OK;
}
