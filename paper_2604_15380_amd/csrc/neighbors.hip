// Radius graph of a batch of structures on gfx950.
//
// Edge set (lead model's cutoff radius, Table 5; periodic systems keep every
// image within the cutoff): (i <- j, n) with
//   t = (n0*a + n1*b) + n2*c,  r = (x_j - x_i) + t,  d2 = (rx*rx + ry*ry) + rz*rz < rc*rc,
// evaluated in IEEE FP64 in that order with contraction disabled, so the set
// is bit-exact.  One wavefront owns one receiver atom and tests candidates
// 64 at a time: a ballot of the hits, a popcount for the count pass and a lane
// prefix for the write position in the fill pass.  The CSR is sorted by
// (receiver, sender, shift).
//
// Candidates come from one of two enumerations, both tested by the same
// expression, so they give the same set:
//  - all pairs: every (j, image) of the structure in sorted order (sender
//    ascending, then (n0, n1, n2) lexicographic), so the compacted hits come
//    out sorted.  Used for small structures and small periodic cells (fewer
//    than 3 bins of width r_c on a periodic axis), i.e. every structure of
//    tens to a few hundred atoms.
//  - cell list: atoms are counting-sorted into bins at least r_c wide and a
//    receiver tests the atoms of the 27 bins around its own.  With >= 3 bins
//    per periodic axis a sender appears at most once per receiver, so the
//    fill pass collects the hits in LDS and ranks them by (sender, shift).
//    A receiver with more hits than that buffer holds is filled by the
//    all-pairs enumeration instead.
#include "internal.h"

namespace {

constexpr int WAVE = 64;

__device__ inline unsigned long long ballot(bool p) { return __ballot(p); }

// per-structure preparation: validation, copies, image range, cell grid ----
constexpr int CELL_MIN_BINS = 64;      // fewer bins: all pairs is as cheap
constexpr double CELL_MARGIN = 1e-9;   // bins are r_c (1 + margin) wide or more

// Shrink a grid to at most `cap` bins by halving its largest axis (bins only
// get wider); axes stay >= lo.
__device__ inline void cap_bins(int nb[3], long long cap, int lo) {
  for (int it = 0; it < 64; ++it) {
    if ((long long)nb[0] * nb[1] * nb[2] <= cap) return;
    int k = nb[0] >= nb[1] ? (nb[0] >= nb[2] ? 0 : 2) : (nb[1] >= nb[2] ? 1 : 2);
    if (nb[k] <= lo) return;
    nb[k] = max(lo, nb[k] / 2);
  }
}

__global__ void __launch_bounds__(256) k_prep(int B, int N, const int32_t* __restrict__ struct_ptr,
                                             const double* __restrict__ pos,
                                             const int32_t* __restrict__ species,
                                             const double* __restrict__ cell,
                                             const uint8_t* __restrict__ pbc, double cutoff,
                                             painn_graph g) {
#pragma clang fp contract(off)
  const int lane = threadIdx.x % WAVE;
  const int b = blockIdx.x * (blockDim.x / WAVE) + threadIdx.x / WAVE;
  if (b >= B) return;
  DevStatus* st = g.d_status;
  int lo = struct_ptr[b], hi = struct_ptr[b + 1];
  bool bad = lo < 0 || hi < lo || hi > N || (b == 0 && lo != 0) || (b == B - 1 && hi != N);
  CellGrid cg{};
  if (bad) {
    if (lane == 0) {
      atomicOr(&st->err, ERR_STRUCT_PTR);
      StructInfo si{};
      si.nimg = 1;
      g.sinfo[b] = si;
      g.grid[b] = cg;
    }
    return;
  }
  if (lane == 0) g.struct_ptr[b] = lo;
  if (lane == 0 && b == B - 1) g.struct_ptr[B] = hi;
  int p[3] = {0, 0, 0};
  double A[9];
  for (int k = 0; k < 9; ++k) A[k] = 0.0;
  if (pbc) {
    for (int k = 0; k < 3; ++k) p[k] = pbc[3 * b + k] != 0;
  }
  const bool periodic = p[0] | p[1] | p[2];
  if (periodic)
    for (int k = 0; k < 9; ++k) A[k] = cell[9 * b + k];
  // copy atoms, species range, Cartesian bounding box
  int smin = 0x7fffffff, smax = -0x7fffffff - 1;
  double xmin[3] = {1e300, 1e300, 1e300}, xmax[3] = {-1e300, -1e300, -1e300};
  for (int i = lo + lane; i < hi; i += WAVE) {
    g.atom_struct[i] = b;
    for (int k = 0; k < 3; ++k) {
      const double x = pos[3 * i + k];
      g.pos[3 * i + k] = x;
      xmin[k] = xmin[k] < x ? xmin[k] : x;
      xmax[k] = xmax[k] > x ? xmax[k] : x;
    }
    int z = species[i];
    g.species[i] = z;
    smin = min(smin, z);
    smax = max(smax, z);
  }
  for (int o = WAVE / 2; o > 0; o /= 2) {
    smin = min(smin, __shfl_xor(smin, o));
    smax = max(smax, __shfl_xor(smax, o));
    for (int k = 0; k < 3; ++k) {
      const double a = __shfl_xor(xmin[k], o), c = __shfl_xor(xmax[k], o);
      xmin[k] = xmin[k] < a ? xmin[k] : a;
      xmax[k] = xmax[k] > c ? xmax[k] : c;
    }
  }
  if (lane == 0 && hi > lo) {
    // every structure's wave reports to the same two words: read first and
    // add to the contention only when the bound moves (the reads may be
    // stale, which only costs an atomic that changes nothing)
    if (smin < __hip_atomic_load(&st->species_min, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
      atomicMin(&st->species_min, smin);
    if (smax > __hip_atomic_load(&st->species_max, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
      atomicMax(&st->species_max, smax);
  }
  const int n = hi - lo;
  const double bin_w = cutoff * (1.0 + CELL_MARGIN);
  const long long bin_cap = 2LL * n + 27;
  int m[3] = {0, 0, 0};
  double frs[9] = {0, 0, 0, 0, 0, 0, 0, 0, 0}, fmn[3] = {0, 0, 0}, fmx[3] = {0, 0, 0}, rwv[3] = {0, 0, 0};
  if (periodic) {
    // reciprocal rows: f_k = x . (a_{k+1} x a_{k+2}) / det
    double cr[9];
    for (int k = 0; k < 3; ++k) {
      const double* u = A + 3 * ((k + 1) % 3);
      const double* v = A + 3 * ((k + 2) % 3);
      cr[3 * k + 0] = u[1] * v[2] - u[2] * v[1];
      cr[3 * k + 1] = u[2] * v[0] - u[0] * v[2];
      cr[3 * k + 2] = u[0] * v[1] - u[1] * v[0];
    }
    double det = A[0] * cr[0] + A[1] * cr[1] + A[2] * cr[2];
    bool ok = isfinite(det) && det != 0.0;
    double fmin[3] = {1e300, 1e300, 1e300}, fmax[3] = {-1e300, -1e300, -1e300};
    for (int i = lo + lane; i < hi && ok; i += WAVE) {
      double x = pos[3 * i], y = pos[3 * i + 1], z = pos[3 * i + 2];
      for (int k = 0; k < 3; ++k) {
        double f = (x * cr[3 * k] + y * cr[3 * k + 1] + z * cr[3 * k + 2]) / det;
        fmin[k] = fmin[k] < f ? fmin[k] : f;
        fmax[k] = fmax[k] > f ? fmax[k] : f;
      }
    }
    for (int k = 0; k < 3; ++k)
      for (int o = WAVE / 2; o > 0; o /= 2) {
        double a = __shfl_xor(fmin[k], o), c = __shfl_xor(fmax[k], o);
        fmin[k] = fmin[k] < a ? fmin[k] : a;
        fmax[k] = fmax[k] > c ? fmax[k] : c;
      }
    long long nimg = 1;
    double w[3] = {0.0, 0.0, 0.0};
    for (int k = 0; k < 3 && ok; ++k) {
      double area = sqrt(cr[3 * k] * cr[3 * k] + cr[3 * k + 1] * cr[3 * k + 1] + cr[3 * k + 2] * cr[3 * k + 2]);
      w[k] = fabs(det) / area;                  // perpendicular width along axis k
      if (!p[k]) continue;
      double span = hi > lo ? fmax[k] - fmin[k] : 0.0;
      // |n_k| < rc / w + |f_j - f_i| for any neighbour image
      double x = cutoff / w[k] + span + 1e-6;
      if (!(x < 127.0)) {
        if (lane == 0) atomicOr(&st->err, ERR_IMAGES);
        ok = false;
        break;
      }
      m[k] = (int)floor(x);
      nimg *= 2 * m[k] + 1;
    }
    if (ok)
      for (int k = 0; k < 3; ++k) {
        for (int c = 0; c < 3; ++c) frs[3 * k + c] = cr[3 * k + c] / det;
        fmn[k] = hi > lo ? fmin[k] : 0.0;
        fmx[k] = hi > lo ? fmax[k] : 0.0;
        rwv[k] = cutoff / w[k];
      }
    if (!ok) {
      if (lane == 0 && !(isfinite(det) && det != 0.0)) atomicOr(&st->err, ERR_CELL);
      m[0] = m[1] = m[2] = 0;
    } else if (nimg * (long long)(hi - lo) >= 0x7fffffffLL) {
      if (lane == 0) atomicOr(&st->err, ERR_IMAGES);
      m[0] = m[1] = m[2] = 0;
    } else if (p[0] && p[1] && p[2] && n > 0) {
      // periodic cell list: >= 3 bins of width >= r_c on every axis; shifts
      // n = q - m_j + m_i stay small when the structure spans few cells
      int nb[3];
      bool use = true;
      for (int k = 0; k < 3; ++k) {
        const double x = floor(w[k] / bin_w);
        nb[k] = x > 1024.0 ? 1024 : (int)x;
        use &= nb[k] >= 3 && fmax[k] - fmin[k] < 64.0 && fabs(fmin[k]) < 1e6 && fabs(fmax[k]) < 1e6;
      }
      if (use) {
        cap_bins(nb, bin_cap, 3);
        if ((long long)nb[0] * nb[1] * nb[2] >= CELL_MIN_BINS) {
          for (int k = 0; k < 3; ++k) {
            cg.nb[k] = nb[k];
            cg.s[k] = (double)nb[k];
            for (int c = 0; c < 3; ++c) cg.fr[3 * k + c] = cr[3 * k + c] / det;
          }
          cg.periodic = 1;
        }
      }
    }
  } else if (n > 0) {
    // molecule cell list over the bounding box
    int nb[3];
    for (int k = 0; k < 3; ++k) {
      const double x = floor((xmax[k] - xmin[k]) / bin_w);
      nb[k] = x < 1.0 ? 1 : (x > 1024.0 ? 1024 : (int)x);
    }
    cap_bins(nb, bin_cap, 1);
    if ((long long)nb[0] * nb[1] * nb[2] >= CELL_MIN_BINS) {
      for (int k = 0; k < 3; ++k) {
        const double ext = xmax[k] - xmin[k];
        cg.nb[k] = nb[k];
        cg.o[k] = xmin[k];
        cg.s[k] = ext > 0.0 ? nb[k] / ext : 0.0;
      }
    }
  }
  if (lane == 0) {
    StructInfo si;
    si.lo = lo;
    si.n = hi - lo;
    si.m0 = m[0];
    si.m1 = m[1];
    si.m2 = m[2];
    si.nimg = (2 * m[0] + 1) * (2 * m[1] + 1) * (2 * m[2] + 1);
    for (int k = 0; k < 9; ++k) si.fr[k] = frs[k];
    for (int k = 0; k < 3; ++k) {
      si.fmin[k] = fmn[k];
      si.fmax[k] = fmx[k];
      si.rw[k] = rwv[k];
    }
    g.sinfo[b] = si;
    for (int k = 0; k < 9; ++k) g.cell[9 * b + k] = A[k];
    cg.base = 2 * lo + 27 * b;
    g.grid[b] = cg;
    if (cg.nb[0] > 0) atomicAdd(&st->cells, 1);
  }
}

__global__ void k_status_init(DevStatus* st) {
  st->n_edges = 0;
  st->err = 0;
  st->species_min = 0x7fffffff;
  st->species_max = -0x7fffffff - 1;
  st->cells = 0;
  st->n_edges_cap = 0;
}

// The image shifts receiver i can need: along a periodic axis k, a pair at
// shift n_k is at least |f_j - f_i + n_k| w_k apart, so only n_k with
// f_i - fmax_k - r_c / w_k < n_k < f_i - fmin_k + r_c / w_k can hold a
// neighbour (widened by 1e-6; n_k = 0 always qualifies).  The box keeps the
// shifts' order, so the rows come out as with the full image range.
struct ImageBox {
  int lo[3], s1, s2, nimg;
};

__device__ inline ImageBox image_box(const StructInfo& si, double xi, double yi, double zi) {
#pragma clang fp contract(off)
  const int m[3] = {si.m0, si.m1, si.m2};
  int lo[3], hi[3];
  for (int k = 0; k < 3; ++k) {
    lo[k] = hi[k] = 0;
    if (m[k] == 0) continue;
    const double f = (xi * si.fr[3 * k] + yi * si.fr[3 * k + 1]) + zi * si.fr[3 * k + 2];
    const double a = f - si.fmax[k] - si.rw[k] - 1e-6, b = f - si.fmin[k] + si.rw[k] + 1e-6;
    lo[k] = a > (double)-m[k] ? min(0, (int)ceil(a)) : -m[k];
    hi[k] = b < (double)m[k] ? max(0, (int)floor(b)) : m[k];
  }
  ImageBox ib;
  ib.lo[0] = lo[0];
  ib.lo[1] = lo[1];
  ib.lo[2] = lo[2];
  ib.s1 = hi[1] - lo[1] + 1;
  ib.s2 = hi[2] - lo[2] + 1;
  ib.nimg = (hi[0] - lo[0] + 1) * ib.s1 * ib.s2;
  return ib;
}

// The candidate test shared by the count and fill passes.  Candidate index t
// enumerates (j, image) with j = lo + t / nimg and image = t % nimg over the
// receiver's image box.
struct Candidate {
  bool hit, zero;
  int j, packed;
};

__device__ inline Candidate test_candidate(int t, int total, int i, const StructInfo& si, const ImageBox& ib,
                                           const double* __restrict__ P, const double* A,
                                           double xi, double yi, double zi, double rc2) {
#pragma clang fp contract(off)
  Candidate c{false, false, 0, 0};
  if (t >= total) return c;
  const int s1 = ib.s1, s2 = ib.s2;
  const int jl = t / ib.nimg;
  const int img = t - jl * ib.nimg;
  const int n0 = img / (s1 * s2) + ib.lo[0];
  const int rem = img % (s1 * s2);
  const int n1 = rem / s2 + ib.lo[1];
  const int n2 = rem % s2 + ib.lo[2];
  const int j = si.lo + jl;
  const double f0 = (double)n0, f1 = (double)n1, f2 = (double)n2;
  const double tx = (f0 * A[0] + f1 * A[3]) + f2 * A[6];
  const double ty = (f0 * A[1] + f1 * A[4]) + f2 * A[7];
  const double tz = (f0 * A[2] + f1 * A[5]) + f2 * A[8];
  const double rx = (P[3 * j + 0] - xi) + tx;
  const double ry = (P[3 * j + 1] - yi) + ty;
  const double rz = (P[3 * j + 2] - zi) + tz;
  const double d2 = (rx * rx + ry * ry) + rz * rz;
  const bool self = (j == i) && (n0 == 0) && (n1 == 0) && (n2 == 0);
  c.hit = !self && d2 < rc2;
  c.zero = !self && d2 == 0.0;
  c.j = j;
  c.packed = (int)((uint32_t)(uint8_t)(int8_t)n0 | ((uint32_t)(uint8_t)(int8_t)n1 << 8) |
                   ((uint32_t)(uint8_t)(int8_t)n2 << 16));
  return c;
}

// The same test for an explicit (j, n) candidate of the cell-list search.
__device__ inline Candidate test_pair(bool valid, int i, int j, int n0, int n1, int n2, const double* __restrict__ P,
                                      const double* A, double xi, double yi, double zi, double rc2) {
#pragma clang fp contract(off)
  Candidate c{false, false, j, 0};
  if (!valid) return c;
  const double f0 = (double)n0, f1 = (double)n1, f2 = (double)n2;
  const double tx = (f0 * A[0] + f1 * A[3]) + f2 * A[6];
  const double ty = (f0 * A[1] + f1 * A[4]) + f2 * A[7];
  const double tz = (f0 * A[2] + f1 * A[5]) + f2 * A[8];
  const double rx = (P[3 * j + 0] - xi) + tx;
  const double ry = (P[3 * j + 1] - yi) + ty;
  const double rz = (P[3 * j + 2] - zi) + tz;
  const double d2 = (rx * rx + ry * ry) + rz * rz;
  const bool self = (j == i) && (n0 == 0) && (n1 == 0) && (n2 == 0);
  c.hit = !self && d2 < rc2;
  c.zero = !self && d2 == 0.0;
  c.packed = (int)((uint32_t)(uint8_t)(int8_t)n0 | ((uint32_t)(uint8_t)(int8_t)n1 << 8) |
                   ((uint32_t)(uint8_t)(int8_t)n2 << 16));
  return c;
}

// Sort key of a packed shift: (n0, n1, n2) lexicographic as an unsigned int.
__device__ inline uint32_t shift_key(int packed) {
  const uint32_t u = (uint32_t)packed;
  return (((u & 0xffu) ^ 0x80u) << 16) | ((((u >> 8) & 0xffu) ^ 0x80u) << 8) | (((u >> 16) & 0xffu) ^ 0x80u);
}

// Cell-list candidates of receiver i: the atoms of the 27 bins around its own
// (clipped at a molecule's bounding box, wrapped with image shift q in a
// periodic cell).  Lane k < 27 owns stencil bin k; `visit(valid, j, n0, n1,
// n2)` is called for 64 candidates at a time by the whole wave.
template <class Visit>
__device__ inline void cell_candidates(const painn_graph& g, const CellGrid& cg, int i, int lane, Visit&& visit) {
  const int local = g.bin_of[i] - cg.base;
  const int c2 = local % cg.nb[2], c1 = (local / cg.nb[2]) % cg.nb[1], c0 = local / (cg.nb[1] * cg.nb[2]);
  int start = 0, cnt = 0, qpk = 0;
  if (lane < 27) {
    int t[3] = {c0 + lane / 9 - 1, c1 + (lane / 3) % 3 - 1, c2 + lane % 3 - 1};
    int q[3] = {0, 0, 0};
    bool ok = true;
    for (int k = 0; k < 3; ++k) {
      if (cg.periodic) {
        q[k] = t[k] < 0 ? -1 : (t[k] >= cg.nb[k] ? 1 : 0);
        t[k] -= q[k] * cg.nb[k];
      } else {
        ok &= t[k] >= 0 && t[k] < cg.nb[k];
      }
    }
    if (ok) {
      const int bin = cg.base + (t[0] * cg.nb[1] + t[1]) * cg.nb[2] + t[2];
      start = g.bin_start[bin];
      cnt = g.bin_start[bin + 1] - start;
      qpk = (q[0] + 1) | ((q[1] + 1) << 2) | ((q[2] + 1) << 4);
    }
  }
  // exclusive prefix of the bin sizes over lanes 0..26
  int incl = cnt;
  for (int o = 1; o < 32; o <<= 1) {
    const int y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  const int excl = incl - cnt;
  const int total = __shfl(incl, 26);
  const int mi0 = g.wrap[3 * i], mi1 = g.wrap[3 * i + 1], mi2 = g.wrap[3 * i + 2];
  for (int t0 = 0; t0 < total; t0 += WAVE) {
    const int t = t0 + lane;
    const bool valid = t < total;
    // stencil slot of candidate t: the last non-empty bin whose prefix is <= t
    int k = 0;
    for (int s = 1; s < 27; ++s)
      if (t >= __builtin_amdgcn_readlane(excl, s) && __builtin_amdgcn_readlane(cnt, s) > 0) k = s;
    const int sk = __shfl(start, k), ek = __shfl(excl, k), qk = __shfl(qpk, k);
    const int j = valid ? g.bin_atoms[sk + (t - ek)] : i;
    int n0 = 0, n1 = 0, n2 = 0;
    if (cg.periodic && valid) {
      n0 = (qk & 3) - 1 - g.wrap[3 * j] + mi0;
      n1 = ((qk >> 2) & 3) - 1 - g.wrap[3 * j + 1] + mi1;
      n2 = ((qk >> 4) & 3) - 1 - g.wrap[3 * j + 2] + mi2;
    }
    visit(valid, j, n0, n1, n2);
  }
}

constexpr int CELL_CAP = 256;   // hits a fill-pass wave ranks in LDS

template <bool FILL>
__global__ void __launch_bounds__(256) k_edges(painn_graph g, double rc2) {
  const int lane = threadIdx.x % WAVE;
  const int wv = threadIdx.x / WAVE;
  const int i = blockIdx.x * (blockDim.x / WAVE) + wv;
  if (i >= g.N) return;
  // atom_struct is only trustworthy when struct_ptr was valid; that error is
  // read back after this pass, so clamp and range-check to stay in bounds.
  int b = g.atom_struct[i];
  b = b < 0 ? 0 : (b >= g.B ? g.B - 1 : b);
  const StructInfo si = g.sinfo[b];
  if (i < si.lo || i >= si.lo + si.n) {
    if (!FILL && lane == 0) g.counts[i] = 0;
    return;
  }
  double A[9];
  for (int k = 0; k < 9; ++k) A[k] = g.cell[9 * b + k];
  const double xi = g.pos[3 * i], yi = g.pos[3 * i + 1], zi = g.pos[3 * i + 2];
  const CellGrid cg = g.grid[b];
  const int out0 = FILL ? g.row_ptr[i] : 0;
  const int deg = FILL ? g.row_ptr[i + 1] - out0 : 0;
  if (cg.nb[0] > 0 && (!FILL || deg <= CELL_CAP)) {
    if (!FILL) {
      int cnt = 0;
      bool zero = false;
      cell_candidates(g, cg, i, lane, [&](bool valid, int j, int n0, int n1, int n2) {
        const Candidate c = test_pair(valid, i, j, n0, n1, n2, g.pos, A, xi, yi, zi, rc2);
        cnt += __popcll(ballot(c.hit));
        zero |= c.zero;
      });
      if (ballot(zero) != 0ull && lane == 0) atomicOr(&g.d_status->err, ERR_COINCIDENT);
      if (lane == 0) g.counts[i] = cnt;
    } else {
      // collect the hits, then place each at its rank by (sender, shift)
      __shared__ int hj[4][CELL_CAP];
      __shared__ int hs[4][CELL_CAP];
      int nh = 0;
      cell_candidates(g, cg, i, lane, [&](bool valid, int j, int n0, int n1, int n2) {
        const Candidate c = test_pair(valid, i, j, n0, n1, n2, g.pos, A, xi, yi, zi, rc2);
        const unsigned long long mask = ballot(c.hit);
        const int at = nh + __popcll(mask & ((1ull << lane) - 1ull));
        if (c.hit && at < CELL_CAP) {
          hj[wv][at] = c.j;
          hs[wv][at] = c.packed;
        }
        nh += __popcll(mask);
      });
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      nh = min(nh, deg);
      for (int e = lane; e < nh; e += WAVE) {
        const int key = hj[wv][e];
        const uint32_t skey = shift_key(hs[wv][e]);
        int rank = 0;
        for (int f = 0; f < nh; ++f) {
          const int kf = hj[wv][f];
          rank += kf < key || (kf == key && shift_key(hs[wv][f]) < skey);
        }
        g.col[out0 + rank] = key;
        g.shift[out0 + rank] = hs[wv][e];
        g.recv[out0 + rank] = i;
      }
    }
    return;
  }
  const ImageBox ib = image_box(si, xi, yi, zi);
  const int total = si.n * ib.nimg;
  int out = out0;
  int cnt = 0;
  bool zero = false;
  for (int t0 = 0; t0 < total; t0 += WAVE) {
    Candidate c = test_candidate(t0 + lane, total, i, si, ib, g.pos, A, xi, yi, zi, rc2);
    unsigned long long mask = ballot(c.hit);
    if (FILL) {
      if (c.hit) {
        int pre = __popcll(mask & ((1ull << lane) - 1ull));
        g.col[out + pre] = c.j;
        g.shift[out + pre] = c.packed;
        g.recv[out + pre] = i;
      }
      out += __popcll(mask);
    } else {
      cnt += __popcll(mask);
      zero |= c.zero;
    }
  }
  if (!FILL) {
    if (ballot(zero) != 0ull && lane == 0) atomicOr(&g.d_status->err, ERR_COINCIDENT);
    if (lane == 0) g.counts[i] = cnt;
  }
}

// ------------------------------------------------------------ binning ----
// Every kernel here returns at once when no structure of the batch uses a
// cell list (st->cells == 0).
__global__ void __launch_bounds__(256) k_bin_clear(long long n, int32_t* __restrict__ cnt, const DevStatus* st) {
  if (st->cells == 0) return;
  for (long long x = (long long)blockIdx.x * 256 + threadIdx.x; x < n; x += (long long)gridDim.x * 256) cnt[x] = 0;
}

// bin of every atom of a cell-list structure, and its fractional floor
__global__ void __launch_bounds__(256) k_bin_assign(painn_graph g) {
#pragma clang fp contract(off)
  if (g.d_status->cells == 0) return;
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= g.N) return;
  int b = g.atom_struct[i];
  b = b < 0 ? 0 : (b >= g.B ? g.B - 1 : b);
  const CellGrid cg = g.grid[b];
  if (cg.nb[0] == 0) return;
  const double x[3] = {g.pos[3 * i], g.pos[3 * i + 1], g.pos[3 * i + 2]};
  int c[3], mw[3] = {0, 0, 0};
  for (int k = 0; k < 3; ++k) {
    double u;
    if (cg.periodic) {
      const double f = (x[0] * cg.fr[3 * k] + x[1] * cg.fr[3 * k + 1]) + x[2] * cg.fr[3 * k + 2];
      const double fl = floor(f);
      mw[k] = (int)fl;
      u = (f - fl) * cg.s[k];
    } else {
      u = (x[k] - cg.o[k]) * cg.s[k];
    }
    const double cu = floor(u);
    c[k] = cu < 0.0 ? 0 : (cu >= (double)cg.nb[k] ? cg.nb[k] - 1 : (int)cu);
  }
  const int bin = cg.base + (c[0] * cg.nb[1] + c[1]) * cg.nb[2] + c[2];
  g.bin_of[i] = bin;
  g.wrap[3 * i] = mw[0];
  g.wrap[3 * i + 1] = mw[1];
  g.wrap[3 * i + 2] = mw[2];
  atomicAdd(&g.bin_count[bin], 1);
}

// atoms into their bins (order within a bin is free: the fill pass ranks);
// the counts return to zero
__global__ void __launch_bounds__(256) k_bin_fill(painn_graph g) {
  if (g.d_status->cells == 0) return;
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= g.N) return;
  int b = g.atom_struct[i];
  b = b < 0 ? 0 : (b >= g.B ? g.B - 1 : b);
  if (g.grid[b].nb[0] == 0) return;
  const int bin = g.bin_of[i];
  const int at = g.bin_start[bin] + atomicSub(&g.bin_count[bin], 1) - 1;
  g.bin_atoms[at] = i;
}

// exclusive scan of n counts -> out[0..n] (1024 elements per block) ---------
// Two uses: per-receiver edge counts -> row_ptr (EDGES: the total is the
// edge count, checked against 2^31 - 1), and per-bin atom counts -> bin
// starts (skipped when no structure uses a cell list).
template <bool EDGES>
__global__ void __launch_bounds__(256) k_scan_blocks(long long n, const int32_t* __restrict__ counts,
                                                    long long* __restrict__ bsum, const DevStatus* st) {
  if (!EDGES && st->cells == 0) return;
  __shared__ long long sh[256];
  const long long base = (long long)blockIdx.x * 1024 + threadIdx.x * 4;
  long long s = 0;
  for (int k = 0; k < 4; ++k)
    if (base + k < n) s += counts[base + k];
  sh[threadIdx.x] = s;
  __syncthreads();
  for (int o = 128; o > 0; o /= 2) {
    if (threadIdx.x < o) sh[threadIdx.x] += sh[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) bsum[blockIdx.x] = sh[0];
}

template <bool EDGES, bool CAPPED = false>
__global__ void __launch_bounds__(256) k_scan_top(int nblk, long long* __restrict__ bsum,
                                                 DevStatus* st, int32_t* __restrict__ out,
                                                 long long n) {
  if (!EDGES && st->cells == 0) return;
  __shared__ long long sh[256];
  long long carry = 0;
  for (int c0 = 0; c0 < nblk; c0 += 256) {
    const int k = c0 + threadIdx.x;
    long long x = k < nblk ? bsum[k] : 0;
    sh[threadIdx.x] = x;
    __syncthreads();
    for (int o = 1; o < 256; o *= 2) {      // inclusive Hillis-Steele scan
      long long y = threadIdx.x >= o ? sh[threadIdx.x - o] : 0;
      __syncthreads();
      sh[threadIdx.x] += y;
      __syncthreads();
    }
    if (k < nblk) bsum[k] = carry + sh[threadIdx.x] - x;   // exclusive
    carry += sh[255];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    if (EDGES && CAPPED) {
      st->n_edges_cap = carry;
    } else if (EDGES) {
      st->n_edges = carry;
      if (carry > 0x7fffffffLL) atomicOr(&st->err, ERR_EDGES);
    }
    out[n] = (int32_t)carry;
  }
}

template <bool EDGES>
__global__ void __launch_bounds__(256) k_scan_apply(long long n, const int32_t* __restrict__ counts,
                                                   const long long* __restrict__ bsum,
                                                   int32_t* __restrict__ out, const DevStatus* st) {
  if (!EDGES && st->cells == 0) return;
  __shared__ long long sh[256];
  const long long base = (long long)blockIdx.x * 1024 + threadIdx.x * 4;
  long long v[4];
  long long s = 0;
  for (int k = 0; k < 4; ++k) {
    v[k] = base + k < n ? counts[base + k] : 0;
    s += v[k];
  }
  sh[threadIdx.x] = s;
  __syncthreads();
  for (int o = 1; o < 256; o *= 2) {
    long long y = threadIdx.x >= o ? sh[threadIdx.x - o] : 0;
    __syncthreads();
    sh[threadIdx.x] += y;
    __syncthreads();
  }
  long long run = bsum[blockIdx.x] + sh[threadIdx.x] - s;
  for (int k = 0; k < 4; ++k) {
    if (base + k < n) out[base + k] = (int32_t)run;
    run += v[k];
  }
}

// ---------------------------------------------------------- neighbour cap ----
__global__ void __launch_bounds__(256) k_cap_counts(int N, int cap, const int32_t* __restrict__ counts,
                                                   int32_t* __restrict__ counts_cap) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < N) counts_cap[i] = min(counts[i], cap);
}

// Squared length of edge (i <- j, packed shift) by the neighbour test's
// exact expression.
__device__ inline double edge_d2(const painn_graph& g, int i, int j, int packed) {
#pragma clang fp contract(off)
  int b = g.atom_struct[i];
  b = b < 0 ? 0 : (b >= g.B ? g.B - 1 : b);
  const double* A = g.cell + 9 * b;
  const double f0 = (double)(int8_t)(packed & 0xff), f1 = (double)(int8_t)((packed >> 8) & 0xff),
               f2 = (double)(int8_t)((packed >> 16) & 0xff);
  const double tx = (f0 * A[0] + f1 * A[3]) + f2 * A[6];
  const double ty = (f0 * A[1] + f1 * A[4]) + f2 * A[7];
  const double tz = (f0 * A[2] + f1 * A[5]) + f2 * A[8];
  const double rx = (g.pos[3 * j + 0] - g.pos[3 * i + 0]) + tx;
  const double ry = (g.pos[3 * j + 1] - g.pos[3 * i + 1]) + ty;
  const double rz = (g.pos[3 * j + 2] - g.pos[3 * i + 2]) + tz;
  return (rx * rx + ry * ry) + rz * rz;
}

// (d2, sender, shift) order; keys within a row are distinct
__device__ inline bool cap_less(double da, int ja, uint32_t sa, double db, int jb, uint32_t sb) {
  return da < db || (da == db && (ja < jb || (ja == jb && sa < sb)));
}

constexpr int CAP_LDS = 256;   // edges of a row a wave ranks from LDS

// Each receiver (one wave) keeps the max_neighbors edges of its full row
// smallest in (d2, sender, shift) and writes them, in row order (sender,
// shift), to its capped row.  Rows longer than CAP_LDS recompute the keys.
__global__ void __launch_bounds__(256) k_cap_select(painn_graph g) {
  __shared__ double kd[4][CAP_LDS];
  __shared__ int kj[4][CAP_LDS];
  __shared__ uint32_t ks[4][CAP_LDS];
  const int lane = threadIdx.x % WAVE, wv = threadIdx.x / WAVE;
  const int i = blockIdx.x * 4 + wv;
  if (i >= g.N) return;
  const int a = g.row_ptr_full[i], deg = g.row_ptr_full[i + 1] - a;
  const int out0 = g.row_ptr[i];
  const int cap = g.max_neighbors;
  if (deg <= cap) {
    for (int e = lane; e < deg; e += WAVE) {
      g.col[out0 + e] = g.col_full[a + e];
      g.shift[out0 + e] = g.shift_full[a + e];
      g.recv[out0 + e] = i;
    }
    return;
  }
  const bool lds = deg <= CAP_LDS;
  if (lds) {
    for (int e = lane; e < deg; e += WAVE) {
      const int j = g.col_full[a + e], p = g.shift_full[a + e];
      kd[wv][e] = edge_d2(g, i, j, p);
      kj[wv][e] = j;
      ks[wv][e] = shift_key(p);
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  int out = out0;
  for (int t0 = 0; t0 < deg; t0 += WAVE) {
    const int e = t0 + lane;
    bool keep = false;
    int j = 0, p = 0;
    if (e < deg) {
      j = g.col_full[a + e];
      p = g.shift_full[a + e];
      const double d = lds ? kd[wv][e] : edge_d2(g, i, j, p);
      const uint32_t sk = shift_key(p);
      int rank = 0;
      for (int f = 0; f < deg && rank < cap; ++f) {
        const double df = lds ? kd[wv][f] : edge_d2(g, i, g.col_full[a + f], g.shift_full[a + f]);
        const int jf = lds ? kj[wv][f] : g.col_full[a + f];
        const uint32_t sf = lds ? ks[wv][f] : shift_key(g.shift_full[a + f]);
        rank += cap_less(df, jf, sf, d, j, sk);
      }
      keep = rank < cap;
    }
    const unsigned long long mask = ballot(keep);
    if (keep) {
      const int at = out + __popcll(mask & ((1ull << lane) - 1ull));
      g.col[at] = j;
      g.shift[at] = p;
      g.recv[at] = i;
    }
    out += __popcll(mask);
  }
}

}  // namespace

hipError_t launch_graph_prep(hipStream_t s, Profiler* p, int B, int N, const int32_t* struct_ptr,
                             const double* pos, const int32_t* species, const double* cell,
                             const uint8_t* pbc, double cutoff, painn_graph* g) {
  prof_mark(p, s, KC_GRAPH_PREP, true);
  k_status_init<<<1, 1, 0, s>>>(g->d_status);
  if (B > 0)
    k_prep<<<(B + 3) / 4, 256, 0, s>>>(B, N, struct_ptr, pos, species, cell, pbc, cutoff, *g);
  // cell-list bins (every kernel returns at once when no structure uses them)
  if (N > 0) {
    const long long nb = (long long)g->n_bins;
    const int nblk = (int)((nb + 1023) / 1024);
    const int cblk = (int)((nb + 255) / 256 < 4096 ? (nb + 255) / 256 : 4096);
    k_bin_clear<<<cblk, 256, 0, s>>>(nb, g->bin_count, g->d_status);
    k_bin_assign<<<(N + 255) / 256, 256, 0, s>>>(*g);
    k_scan_blocks<false><<<nblk, 256, 0, s>>>(nb, g->bin_count, g->bin_scan_tmp, g->d_status);
    k_scan_top<false><<<1, 256, 0, s>>>(nblk, g->bin_scan_tmp, g->d_status, g->bin_start, nb);
    k_scan_apply<false><<<nblk, 256, 0, s>>>(nb, g->bin_count, g->bin_scan_tmp, g->bin_start, g->d_status);
    k_bin_fill<<<(N + 255) / 256, 256, 0, s>>>(*g);
  }
  prof_mark(p, s, KC_GRAPH_PREP, false);
  return hipGetLastError();
}

hipError_t launch_graph_count(hipStream_t s, Profiler* p, painn_graph* g) {
  prof_mark(p, s, KC_GRAPH_COUNT, true);
  if (g->N > 0) k_edges<false><<<(g->N + 3) / 4, 256, 0, s>>>(*g, g->cutoff * g->cutoff);
  prof_mark(p, s, KC_GRAPH_COUNT, false);
  return hipGetLastError();
}

hipError_t launch_graph_scan(hipStream_t s, Profiler* p, painn_graph* g) {
  const int nblk = (g->N + 1023) / 1024;
  prof_mark(p, s, KC_GRAPH_SCAN, true);
  if (nblk > 0) k_scan_blocks<true><<<nblk, 256, 0, s>>>(g->N, g->counts, g->scan_tmp, g->d_status);
  k_scan_top<true><<<1, 256, 0, s>>>(nblk, g->scan_tmp, g->d_status, g->row_ptr, g->N);
  if (nblk > 0) k_scan_apply<true><<<nblk, 256, 0, s>>>(g->N, g->counts, g->scan_tmp, g->row_ptr, g->d_status);
  prof_mark(p, s, KC_GRAPH_SCAN, false);
  return hipGetLastError();
}

hipError_t launch_graph_fill(hipStream_t s, Profiler* p, painn_graph* g) {
  prof_mark(p, s, KC_GRAPH_FILL, true);
  if (g->N > 0 && g->E > 0) k_edges<true><<<(g->N + 3) / 4, 256, 0, s>>>(*g, g->cutoff * g->cutoff);
  prof_mark(p, s, KC_GRAPH_FILL, false);
  return hipGetLastError();
}

hipError_t launch_graph_cap_scan(hipStream_t s, Profiler* p, painn_graph* g) {
  const int nblk = (g->N + 1023) / 1024;
  prof_mark(p, s, KC_GRAPH_SCAN, true);
  if (g->N > 0) k_cap_counts<<<(g->N + 255) / 256, 256, 0, s>>>(g->N, g->max_neighbors, g->counts, g->counts_cap);
  if (nblk > 0) k_scan_blocks<true><<<nblk, 256, 0, s>>>(g->N, g->counts_cap, g->scan_tmp, g->d_status);
  k_scan_top<true, true><<<1, 256, 0, s>>>(nblk, g->scan_tmp, g->d_status, g->row_ptr, g->N);
  if (nblk > 0) k_scan_apply<true><<<nblk, 256, 0, s>>>(g->N, g->counts_cap, g->scan_tmp, g->row_ptr, g->d_status);
  prof_mark(p, s, KC_GRAPH_SCAN, false);
  return hipGetLastError();
}

hipError_t launch_graph_cap_select(hipStream_t s, Profiler* p, painn_graph* g) {
  prof_mark(p, s, KC_GRAPH_FILL, true);
  if (g->N > 0 && g->E > 0) k_cap_select<<<(g->N + 3) / 4, 256, 0, s>>>(*g);
  prof_mark(p, s, KC_GRAPH_FILL, false);
  return hipGetLastError();
}
