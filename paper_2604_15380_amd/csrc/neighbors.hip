// Radius graph of a batch of small structures on gfx950.
//
// Edge set (lead model's cutoff radius, Table 5; periodic systems keep every
// image within the cutoff): (i <- j, n) with
//   t = (n0*a + n1*b) + n2*c,  r = (x_j - x_i) + t,  d2 = (rx*rx + ry*ry) + rz*rz < rc*rc,
// evaluated in IEEE FP64 in that order with contraction disabled, so the set
// is bit-exact.  One wavefront owns one receiver atom and walks the candidate
// list (sender j ascending, then image index ascending = (n0, n1, n2)
// lexicographic) 64 candidates at a time: a ballot of the hits, a popcount for
// the count pass and a lane prefix (mbcnt) for the write position in the fill
// pass.  Because candidates are visited in sorted order, the CSR comes out
// sorted by (receiver, sender, shift) with no sort step.
//
// Structures here are small (tens to a few hundred atoms, up to 125 images),
// so every candidate pair is tested; a cell list pays off only once a cell is
// wider than 3 r_c per axis, which none of these workloads reach.
#include "internal.h"

namespace {

constexpr int WAVE = 64;

__device__ inline unsigned long long ballot(bool p) { return __ballot(p); }

// per-structure preparation: validation, copies, image range --------------
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
  if (bad) {
    if (lane == 0) {
      atomicOr(&st->err, ERR_STRUCT_PTR);
      StructInfo si{0, 0, 0, 0, 0, 1};
      g.sinfo[b] = si;
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
  // copy atoms, species range
  int smin = 0x7fffffff, smax = -0x7fffffff - 1;
  for (int i = lo + lane; i < hi; i += WAVE) {
    g.atom_struct[i] = b;
    g.pos[3 * i + 0] = pos[3 * i + 0];
    g.pos[3 * i + 1] = pos[3 * i + 1];
    g.pos[3 * i + 2] = pos[3 * i + 2];
    int z = species[i];
    g.species[i] = z;
    smin = min(smin, z);
    smax = max(smax, z);
  }
  for (int o = WAVE / 2; o > 0; o /= 2) {
    smin = min(smin, __shfl_xor(smin, o));
    smax = max(smax, __shfl_xor(smax, o));
  }
  if (lane == 0 && hi > lo) {
    atomicMin(&st->species_min, smin);
    atomicMax(&st->species_max, smax);
  }
  int m[3] = {0, 0, 0};
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
    for (int k = 0; k < 3 && ok; ++k) {
      if (!p[k]) continue;
      double area = sqrt(cr[3 * k] * cr[3 * k] + cr[3 * k + 1] * cr[3 * k + 1] + cr[3 * k + 2] * cr[3 * k + 2]);
      double w = fabs(det) / area;              // perpendicular width along axis k
      double span = hi > lo ? fmax[k] - fmin[k] : 0.0;
      // |n_k| < rc / w + |f_j - f_i| for any neighbour image
      double x = cutoff / w + span + 1e-6;
      if (!(x < 127.0)) {
        if (lane == 0) atomicOr(&st->err, ERR_IMAGES);
        ok = false;
        break;
      }
      m[k] = (int)floor(x);
      nimg *= 2 * m[k] + 1;
    }
    if (!ok) {
      if (lane == 0 && !(isfinite(det) && det != 0.0)) atomicOr(&st->err, ERR_CELL);
      m[0] = m[1] = m[2] = 0;
    } else if (nimg * (long long)(hi - lo) >= 0x7fffffffLL) {
      if (lane == 0) atomicOr(&st->err, ERR_IMAGES);
      m[0] = m[1] = m[2] = 0;
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
    g.sinfo[b] = si;
    for (int k = 0; k < 9; ++k) g.cell[9 * b + k] = A[k];
  }
}

__global__ void k_status_init(DevStatus* st) {
  st->n_edges = 0;
  st->err = 0;
  st->species_min = 0x7fffffff;
  st->species_max = -0x7fffffff - 1;
  st->pad = 0;
}

// The candidate test shared by the count and fill passes.  Candidate index t
// enumerates (j, image) with j = lo + t / nimg and image = t % nimg.
struct Candidate {
  bool hit, zero;
  int j, packed;
};

__device__ inline Candidate test_candidate(int t, int total, int i, const StructInfo& si,
                                           const double* __restrict__ P, const double* A,
                                           double xi, double yi, double zi, double rc2) {
#pragma clang fp contract(off)
  Candidate c{false, false, 0, 0};
  if (t >= total) return c;
  const int s1 = 2 * si.m1 + 1, s2 = 2 * si.m2 + 1;
  const int jl = t / si.nimg;
  const int img = t - jl * si.nimg;
  const int n0 = img / (s1 * s2) - si.m0;
  const int rem = img % (s1 * s2);
  const int n1 = rem / s2 - si.m1;
  const int n2 = rem % s2 - si.m2;
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

template <bool FILL>
__global__ void __launch_bounds__(256) k_edges(painn_graph g, double rc2) {
  const int lane = threadIdx.x % WAVE;
  const int i = blockIdx.x * (blockDim.x / WAVE) + threadIdx.x / WAVE;
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
  const int total = si.n * si.nimg;
  int out = FILL ? g.row_ptr[i] : 0;
  int cnt = 0;
  bool zero = false;
  for (int t0 = 0; t0 < total; t0 += WAVE) {
    Candidate c = test_candidate(t0 + lane, total, i, si, g.pos, A, xi, yi, zi, rc2);
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

// exclusive scan of counts -> row_ptr (1024 elements per block) -------------
__global__ void __launch_bounds__(256) k_scan_blocks(int N, const int32_t* __restrict__ counts,
                                                    long long* __restrict__ bsum) {
  __shared__ long long sh[256];
  const int base = blockIdx.x * 1024 + threadIdx.x * 4;
  long long s = 0;
  for (int k = 0; k < 4; ++k)
    if (base + k < N) s += counts[base + k];
  sh[threadIdx.x] = s;
  __syncthreads();
  for (int o = 128; o > 0; o /= 2) {
    if (threadIdx.x < o) sh[threadIdx.x] += sh[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) bsum[blockIdx.x] = sh[0];
}

__global__ void __launch_bounds__(256) k_scan_top(int nblk, long long* __restrict__ bsum,
                                                 DevStatus* st, int32_t* __restrict__ row_ptr,
                                                 int N) {
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
    st->n_edges = carry;
    if (carry > 0x7fffffffLL) atomicOr(&st->err, ERR_EDGES);
    row_ptr[N] = (int32_t)carry;
  }
}

__global__ void __launch_bounds__(256) k_scan_apply(int N, const int32_t* __restrict__ counts,
                                                   const long long* __restrict__ bsum,
                                                   int32_t* __restrict__ row_ptr) {
  __shared__ long long sh[256];
  const int base = blockIdx.x * 1024 + threadIdx.x * 4;
  long long v[4];
  long long s = 0;
  for (int k = 0; k < 4; ++k) {
    v[k] = base + k < N ? counts[base + k] : 0;
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
    if (base + k < N) row_ptr[base + k] = (int32_t)run;
    run += v[k];
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
  if (nblk > 0) k_scan_blocks<<<nblk, 256, 0, s>>>(g->N, g->counts, g->scan_tmp);
  k_scan_top<<<1, 256, 0, s>>>(nblk, g->scan_tmp, g->d_status, g->row_ptr, g->N);
  if (nblk > 0) k_scan_apply<<<nblk, 256, 0, s>>>(g->N, g->counts, g->scan_tmp, g->row_ptr);
  prof_mark(p, s, KC_GRAPH_SCAN, false);
  return hipGetLastError();
}

hipError_t launch_graph_fill(hipStream_t s, Profiler* p, painn_graph* g) {
  prof_mark(p, s, KC_GRAPH_FILL, true);
  if (g->N > 0 && g->E > 0) k_edges<true><<<(g->N + 3) / 4, 256, 0, s>>>(*g, g->cutoff * g->cutoff);
  prof_mark(p, s, KC_GRAPH_FILL, false);
  return hipGetLastError();
}
