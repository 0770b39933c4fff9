// Radius graph of a batch of atomic systems: the edges the layer consumes,
// built on the device (App. "Model and Training Configurations": the graph is
// built on the fly from a cutoff, with a limit on the neighbours per atom).
//
// Edge (src, dst, n): atoms of one system, source image n in {-1,0,1} per
// periodic axis (0 elsewhere), vector r = (pos[src] - pos[dst]) + n * L,
// kept when |r|^2 < r_cut^2 (not the atom itself with n = 0).  The float32
// operations are fixed, each rounded on its own (no fused multiply-add):
// difference, image added, |r|^2 = (rx*rx + ry*ry) + rz*rz, compared with
// r_cut*r_cut, so the edge set and the vectors are exact functions of the
// float32 inputs.  With a cap K, an atom keeps its K candidates smallest in
// (|r|^2, src, image code); edges are ordered by (dst, src, image code),
// code = (nx+1)*9 + (ny+1)*3 + (nz+1).
//
// Cells: every system gets its own grid of cells at least 1.001 r_cut wide
// (at most 1024 per axis and 2 n_g + 1 per system, n_g its atom count; the
// width grows where those bounds bind), over [0, L) on periodic axes and the
// system's bounding box elsewhere.  An atom's neighbours within the cutoff
// then lie in its own or an adjacent cell (the 1.001 margin covers the
// rounding of the cell coordinate, whose error stays below 1024 * 2^-23 cell
// widths); adjacency wraps on periodic axes, the wrap giving the image.  Cell
// ids are system-major (system g's cells start at 2 ptr[g] + g, so no
// prefix sum over systems is needed); atoms are placed in cell order by a
// counting scatter (atomic per-cell counts, their prefix sum, one scatter).
//
// Passes: per-system grids; per-atom cell ids and cell counts; their prefix
// sum; positions in cell order; a count pass (one wave per destination, the
// 27 adjacent cells flattened over the lanes); a prefix sum of the kept
// counts with their maximum; and an emit pass (one wave per destination)
// that gathers the candidates into LDS, sorts them there (bitonic; first by
// (|r|^2, key) when the cap binds) and writes the edges in (src, image)
// order, so the output does not depend on the order of atoms inside a cell.
#include "common.hpp"
#include "kernels.h"

namespace tdn {

namespace {

constexpr float kCellMargin = 1.001f;
constexpr int kMaxCellsPerAxis = 1024;

struct GridParams {  // one system's cell grid (64 bytes)
  float lo[3], inv[3], L[3];
  int n[3];
  int base;
  int pad[3];
};

size_t al(size_t b) { return (b + 255) & ~size_t(255); }

__device__ __forceinline__ bool finite3(float x, float y, float z) {
  return isfinite(x) && isfinite(y) && isfinite(z);
}

// One block per system: bounding box on non-periodic axes, grid size.
__global__ __launch_bounds__(256) void k_rg_grid(RadiusGraphArgs a, GridParams* __restrict__ params,
                                                 int32_t* __restrict__ flags) {
  const int g = blockIdx.x, tid = threadIdx.x;
  int a0 = a.graph_ptr[g], a1 = a.graph_ptr[g + 1];
  const bool bad_ptr = a0 < 0 || a1 < a0 || a1 > a.N || (g == 0 && a0 != 0) || (g == a.G - 1 && a1 != a.N);
  if (bad_ptr) {
    if (tid == 0) atomicOr(&flags[0], 1);
    a0 = min(max(a0, 0), a.N);
    a1 = min(max(a1, a0), a.N);
  }
  __shared__ float red[6][256];
  float mn[3] = {INFINITY, INFINITY, INFINITY}, mx[3] = {-INFINITY, -INFINITY, -INFINITY};
  for (int i = a0 + tid; i < a1; i += 256) {
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      const float v = a.pos[3 * size_t(i) + k];
      mn[k] = fminf(mn[k], v);
      mx[k] = fmaxf(mx[k], v);
    }
  }
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    red[k][tid] = mn[k];
    red[3 + k][tid] = mx[k];
  }
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (tid < off) {
#pragma unroll
      for (int k = 0; k < 3; ++k) {
        red[k][tid] = fminf(red[k][tid], red[k][tid + off]);
        red[3 + k][tid] = fmaxf(red[3 + k][tid], red[3 + k][tid + off]);
      }
    }
    __syncthreads();
  }
  if (tid != 0) return;
  const float rcm = a.r_cut * kCellMargin;
  GridParams P{};
  float ext[3];
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    if (a.periodic[k]) {
      const float L = a.cell[3 * size_t(g) + k];
      if (!(L >= a.r_cut) || !isfinite(L)) atomicOr(&flags[1], 1);
      P.L[k] = L;
      P.lo[k] = 0.f;
      ext[k] = isfinite(L) && L > 0.f ? L : 0.f;
    } else {
      const bool empty = a1 == a0 || !(red[3 + k][0] >= red[k][0]);
      P.L[k] = 0.f;
      P.lo[k] = empty ? 0.f : red[k][0];
      ext[k] = empty ? 0.f : red[3 + k][0] - red[k][0];
      if (!isfinite(ext[k])) ext[k] = 0.f;
    }
    const float q = ext[k] / rcm;
    P.n[k] = q >= float(kMaxCellsPerAxis) ? kMaxCellsPerAxis : max(1, int(q));
  }
  // at most 2 n_g + 1 cells per system: halve the largest axis count
  const int64_t budget = 2 * int64_t(a1 - a0) + 1;
  int nx = P.n[0], ny = P.n[1], nz = P.n[2];
  while (int64_t(nx) * ny * nz > budget) {
    if (nx >= ny && nx >= nz) nx = max(1, nx / 2);
    else if (ny >= nz) ny = max(1, ny / 2);
    else nz = max(1, nz / 2);
  }
  P.n[0] = nx;
  P.n[1] = ny;
  P.n[2] = nz;
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    const float w = a.periodic[k] ? ext[k] / float(P.n[k]) : fmaxf(ext[k] / float(P.n[k]), rcm);
    P.inv[k] = w > 0.f ? 1.f / w : 0.f;
  }
  P.base = 2 * a0 + g;
  params[g] = P;
}

// Cell coordinate of position x on one axis of a grid (clamped into the grid).
__device__ __forceinline__ int cell_coord(float x, float lo, float inv, int n) {
  const float q = (x - lo) * inv;
  const int c = q >= float(n) ? n - 1 : (q > 0.f ? int(q) : 0);  // NaN -> 0
  return min(c, n - 1);
}

// One thread per atom: its system (binary search over graph_ptr), cell id,
// and a slot in the cell (the cell's atom count, zeroed beforehand, counted
// up with atomics: the order inside a cell is arbitrary, which the emit
// pass's sort makes irrelevant).
__global__ __launch_bounds__(256) void k_rg_keys(RadiusGraphArgs a, const GridParams* __restrict__ params,
                                                 int n_keys, int32_t* __restrict__ keys, int32_t* __restrict__ gid,
                                                 int32_t* __restrict__ cell_cnt, int32_t* __restrict__ rank,
                                                 int32_t* __restrict__ flags) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= a.N) return;
  int lo = 0, hi = a.G;  // last g with graph_ptr[g] <= i
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (a.graph_ptr[mid] <= i) lo = mid; else hi = mid;
  }
  const int g = lo;
  const GridParams P = params[g];
  const float x = a.pos[3 * size_t(i)], y = a.pos[3 * size_t(i) + 1], z = a.pos[3 * size_t(i) + 2];
  bool bad = !finite3(x, y, z);
  const float p[3] = {x, y, z};
  int c[3];
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    if (a.periodic[k] && !(p[k] >= 0.f && p[k] < P.L[k])) bad = true;
    c[k] = cell_coord(p[k], P.lo[k], P.inv[k], P.n[k]);
  }
  if (bad) atomicOr(&flags[1], 1);
  const int key = min(max(P.base + (c[2] * P.n[1] + c[1]) * P.n[0] + c[0], 0), n_keys - 1);
  keys[i] = key;
  gid[i] = g;
  rank[i] = atomicAdd(&cell_cnt[key], 1);
}

// Positions in cell order (cell_off: exclusive prefix of the cell counts),
// the atom id in .w.
__global__ __launch_bounds__(256) void k_rg_scatter(int N, const float* __restrict__ pos,
                                                    const int32_t* __restrict__ keys,
                                                    const int32_t* __restrict__ rank,
                                                    const int32_t* __restrict__ cell_off,
                                                    float4* __restrict__ spos) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= N) return;
  const int j = cell_off[keys[i]] + rank[i];
  spos[j] = make_float4(pos[3 * size_t(i)], pos[3 * size_t(i) + 1], pos[3 * size_t(i) + 2], __int_as_float(i));
}

// Everything a destination atom's wave needs to scan its 27 adjacent cells.
struct DstCtx {
  int i;
  float px, py, pz;
  GridParams P;
  int c[3];
};

__device__ __forceinline__ DstCtx dst_ctx(const RadiusGraphArgs& a, const GridParams* __restrict__ params,
                                          const int32_t* __restrict__ keys, const int32_t* __restrict__ gid, int i) {
  DstCtx d;
  d.i = i;
  d.px = a.pos[3 * size_t(i)];
  d.py = a.pos[3 * size_t(i) + 1];
  d.pz = a.pos[3 * size_t(i) + 2];
  d.P = params[gid[i]];
  int local = keys[i] - d.P.base;  // decode the cell id (clamped ids stay in range)
  const int nx = d.P.n[0], ny = d.P.n[1];
  local = max(local, 0);
  d.c[0] = local % nx;
  d.c[1] = (local / nx) % ny;
  d.c[2] = min(local / (nx * ny), d.P.n[2] - 1);
  return d;
}

// Calls visit(hit, key, r2) once per candidate slot of the wave (all lanes
// together, hit false on idle lanes).  The 27 adjacent cells are flattened
// into one slot range: lane k < 27 takes cell k (its atom range, image and
// whether it exists), a lane prefix sum gives each cell's first slot, and
// each slot finds its cell by a five-step search over the prefix.  Wraps on
// periodic axes give the image; cells past a non-periodic edge are empty.
// key = src * 32 + image code.
template <typename Visit>
__device__ __forceinline__ void for_each_candidate(const RadiusGraphArgs& a, const DstCtx& d,
                                                   const int32_t* __restrict__ cell_off, int n_keys,
                                                   const float4* __restrict__ spos, float rc2, int lane,
                                                   Visit&& visit) {
  int beg = 0, cnt = 0, code = 13;
  if (lane < 27) {
    const int o[3] = {lane % 3 - 1, (lane / 3) % 3 - 1, lane / 9 - 1};
    int cc[3], img[3];
    bool skip = false;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      int v = d.c[k] + o[k];
      img[k] = 0;
      if (a.periodic[k]) {
        if (v < 0) { v += d.P.n[k]; img[k] = -1; }
        else if (v >= d.P.n[k]) { v -= d.P.n[k]; img[k] = 1; }
      } else if (v < 0 || v >= d.P.n[k]) {
        skip = true;
      }
      cc[k] = v;
    }
    if (!skip) {
      const int key = min(max(d.P.base + (cc[2] * d.P.n[1] + cc[1]) * d.P.n[0] + cc[0], 0), n_keys - 1);
      beg = cell_off[key];
      cnt = cell_off[key + 1] - beg;
    }
    code = (img[0] + 1) * 9 + (img[1] + 1) * 3 + (img[2] + 1);
  }
  int incl = cnt;
#pragma unroll
  for (int o = 1; o < 32; o <<= 1) {
    const int t = __shfl_up(incl, o);
    if (lane >= o) incl += t;
  }
  const int excl = incl - cnt;
  const int total = __shfl(incl, 26);
  for (int sb = 0; sb < total; sb += kWave) {
    const int slot = sb + lane;
    int c = 0;  // cells before the slot's: lanes k < 27 with incl[k] <= slot
#pragma unroll
    for (int step = 16; step > 0; step >>= 1) {
      const int v = __shfl(incl, min(c + step - 1, 26));
      if (c + step <= 27 && v <= slot) c += step;
    }
    c = min(c, 26);
    const int cb = __shfl(beg, c), ce = __shfl(excl, c), cd = __shfl(code, c);
    bool hit = false;
    uint32_t ekey = 0;
    float r2 = 0.f;
    if (slot < total) {
      const float4 q = spos[cb + (slot - ce)];
      const int src = __float_as_int(q.w);
      const float sx = float(cd / 9 - 1) * d.P.L[0], sy = float((cd / 3) % 3 - 1) * d.P.L[1],
                  sz = float(cd % 3 - 1) * d.P.L[2];
      const float rx = __fadd_rn(__fsub_rn(q.x, d.px), sx);
      const float ry = __fadd_rn(__fsub_rn(q.y, d.py), sy);
      const float rz = __fadd_rn(__fsub_rn(q.z, d.pz), sz);
      r2 = __fadd_rn(__fadd_rn(__fmul_rn(rx, rx), __fmul_rn(ry, ry)), __fmul_rn(rz, rz));
      hit = r2 < rc2 && !(cd == 13 && src == d.i);
      ekey = uint32_t(src) * 32u + uint32_t(cd);
    }
    visit(hit, ekey, r2);
  }
}

// One wave per destination atom: candidates within the cutoff (tot) and the
// edges kept (offs, before the prefix sum).
__global__ __launch_bounds__(256) void k_rg_count(RadiusGraphArgs a, const GridParams* __restrict__ params,
                                                  const int32_t* __restrict__ keys, const int32_t* __restrict__ gid,
                                                  const int32_t* __restrict__ cell_off, int n_keys,
                                                  const float4* __restrict__ spos, float rc2,
                                                  int32_t* __restrict__ offs, int32_t* __restrict__ tot) {
  const int lane = threadIdx.x & (kWave - 1);
  const int i = __builtin_amdgcn_readfirstlane(int(blockIdx.x * 4 + threadIdx.x / kWave));
  if (i >= a.N) return;
  const DstCtx d = dst_ctx(a, params, keys, gid, i);
  int total = 0;
  for_each_candidate(a, d, cell_off, n_keys, spos, rc2, lane,
                     [&](bool hit, uint32_t, float) { total += __popcll(__ballot(hit)); });
  if (lane == 0) {
    offs[i] = a.max_neighbors > 0 ? min(total, a.max_neighbors) : total;
    tot[i] = total;
  }
}

// One workgroup: offs[0..N-1] -> exclusive prefix sum with offs[N] = E, and
// the largest candidate count and the neighbour-limit flag into flags.
__global__ __launch_bounds__(1024) void k_rg_scan(int N, int32_t* __restrict__ offs,
                                                  const int32_t* __restrict__ tot, int32_t* __restrict__ flags) {
  __shared__ int32_t part[1024], pmax[1024];
  const int t = threadIdx.x;
  const int per = (N + 1023) / 1024;
  const int lo = min(N, t * per), hi = min(N, lo + per);
  int32_t sum = 0, mx = 0;
  for (int i = lo; i < hi; ++i) {
    sum += offs[i];
    mx = max(mx, tot[i]);
  }
  part[t] = sum;
  pmax[t] = mx;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    const int32_t v = t >= off ? part[t - off] : 0;
    const int32_t m = t >= off ? pmax[t - off] : 0;
    __syncthreads();
    part[t] += v;
    pmax[t] = max(pmax[t], m);
    __syncthreads();
  }
  int32_t run = part[t] - sum;
  for (int i = lo; i < hi; ++i) {
    const int32_t v = offs[i];
    offs[i] = run;
    run += v;
  }
  if (t == 1023) {
    offs[N] = part[1023];
    flags[4] = pmax[1023];
    flags[2] = pmax[1023] > kRadiusMaxNeighbours;
  }
}

// Ascending bitonic sort of P (a power of two) 64-bit keys in LDS by one
// wave (a workgroup of one wave: the barriers order its LDS traffic).
__device__ __forceinline__ void bitonic_sort(uint64_t* s, int P, int lane) {
  for (int k = 2; k <= P; k <<= 1)
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int t = lane; t < (P >> 1); t += kWave) {
        const int i0 = ((t & ~(j - 1)) << 1) | (t & (j - 1)), i1 = i0 + j;
        const bool up = (i0 & k) == 0;
        const uint64_t x = s[i0], y = s[i1];
        if ((x > y) == up) {
          s[i0] = y;
          s[i1] = x;
        }
      }
      __syncthreads();
    }
}

// One single-wave workgroup per destination atom: gather, order, write.
__global__ __launch_bounds__(kWave) void k_rg_emit(RadiusGraphArgs a, const GridParams* __restrict__ params,
                                                   const int32_t* __restrict__ keys, const int32_t* __restrict__ gid,
                                                   const int32_t* __restrict__ cell_off, int n_keys,
                                                   const float4* __restrict__ spos, float rc2,
                                                   const int32_t* __restrict__ offs, int P,
                                                   int32_t* __restrict__ edge_index, float* __restrict__ edge_vec,
                                                   int32_t* __restrict__ edge_image) {
  extern __shared__ uint64_t sk[];
  const int lane = threadIdx.x;
  const int i = blockIdx.x;
  const int e0 = offs[i], keep = offs[i + 1] - e0, E = offs[a.N];
  const DstCtx d = dst_ctx(a, params, keys, gid, i);
  int n = 0;
  const bool capped = a.max_neighbors > 0;
  for_each_candidate(a, d, cell_off, n_keys, spos, rc2, lane,
                     [&](bool hit, uint32_t key, float r2) {
                       const uint64_t m = __ballot(hit);
                       if (hit) {
                         const int pos = n + __popcll(m & ((1ull << lane) - 1));
                         if (pos < P)
                           sk[pos] = capped ? (uint64_t(__float_as_uint(r2)) << 32) | key : uint64_t(key);
                       }
                       n += __popcll(m);
                     });
  n = min(n, P);
  for (int t = n + lane; t < P; t += kWave) sk[t] = ~0ull;
  __syncthreads();
  bitonic_sort(sk, P, lane);
  if (capped) {
    // the `keep` nearest, then in (src, image) order (|r|^2 >= 0 orders by its bits)
    for (int t = lane; t < P; t += kWave) sk[t] = t < keep ? (sk[t] & 0xffffffffull) : ~0ull;
    __syncthreads();
    bitonic_sort(sk, P, lane);
  }
  // (the count pass found the same n; both guards only keep a disagreement in bounds)
  for (int t = lane; t < min(keep, n); t += kWave) {
    const uint32_t key = uint32_t(sk[t]);
    const int src = int(key >> 5), code = int(key & 31u);
    if (src >= a.N) continue;
    const int img[3] = {code / 9 - 1, (code / 3) % 3 - 1, code % 3 - 1};
    const float rx = __fadd_rn(__fsub_rn(a.pos[3 * size_t(src)], d.px), float(img[0]) * d.P.L[0]);
    const float ry = __fadd_rn(__fsub_rn(a.pos[3 * size_t(src) + 1], d.py), float(img[1]) * d.P.L[1]);
    const float rz = __fadd_rn(__fsub_rn(a.pos[3 * size_t(src) + 2], d.pz), float(img[2]) * d.P.L[2]);
    const size_t e = size_t(e0) + t;
    edge_index[e] = src;
    edge_index[size_t(E) + e] = i;
    edge_vec[3 * e] = rx;
    edge_vec[3 * e + 1] = ry;
    edge_vec[3 * e + 2] = rz;
    if (edge_image) {
      edge_image[3 * e] = img[0];
      edge_image[3 * e + 1] = img[1];
      edge_image[3 * e + 2] = img[2];
    }
  }
}

}  // namespace

RadiusGraphLayout radius_graph_layout(int N, int G) {
  RadiusGraphLayout l{};
  l.n_keys = 2 * N + G;
  size_t o = 0;
  l.params = o; o += al(size_t(G) * sizeof(GridParams));
  l.keys = o; o += al(size_t(N) * 4);
  l.gid = o; o += al(size_t(N) * 4);
  l.rank = o; o += al(size_t(N) * 4);
  l.flags = o; o += 256;  // flags, then the cell counts: cleared together
  l.cell_off = o; o += al((size_t(l.n_keys) + 1) * 4);
  l.spos = o; o += al(size_t(N) * 16);
  l.offs = o; o += al((size_t(N) + 1) * 4);
  l.tot = o; o += al(size_t(N) * 4);
  l.total = o;
  return l;
}

hipError_t launch_radius_count(const RadiusGraphArgs& a, char* ws, hipStream_t s) {
  const RadiusGraphLayout l = radius_graph_layout(a.N, a.G);
  int32_t* flags = reinterpret_cast<int32_t*>(ws + l.flags);
  int32_t* offs = reinterpret_cast<int32_t*>(ws + l.offs);
  if (a.N == 0) {
    hipError_t e = launch_zero(flags, 64, s);
    return e != hipSuccess ? e : launch_zero(offs, 4, s);
  }
  // flags and cell counts are adjacent: one clear
  hipError_t e = launch_zero(flags, 256 + (size_t(l.n_keys) + 1) * 4, s);
  if (e != hipSuccess) return e;
  auto* params = reinterpret_cast<GridParams*>(ws + l.params);
  auto* keys = reinterpret_cast<int32_t*>(ws + l.keys);
  auto* gid = reinterpret_cast<int32_t*>(ws + l.gid);
  auto* rank = reinterpret_cast<int32_t*>(ws + l.rank);
  auto* cell_off = reinterpret_cast<int32_t*>(ws + l.cell_off);
  auto* spos = reinterpret_cast<float4*>(ws + l.spos);
  auto* tot = reinterpret_cast<int32_t*>(ws + l.tot);
  const unsigned nb = unsigned((a.N + 255) / 256);
  k_rg_grid<<<dim3(a.G), dim3(256), 0, s>>>(a, params, flags);
  k_rg_keys<<<dim3(nb), dim3(256), 0, s>>>(a, params, l.n_keys, keys, gid, cell_off, rank, flags);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = launch_scan_exclusive(cell_off, l.n_keys + 1, s);
  if (e != hipSuccess) return e;
  k_rg_scatter<<<dim3(nb), dim3(256), 0, s>>>(a.N, a.pos, keys, rank, cell_off, spos);
  const float rc2 = a.r_cut * a.r_cut;
  k_rg_count<<<dim3(unsigned((a.N + 3) / 4)), dim3(256), 0, s>>>(a, params, keys, gid, cell_off, l.n_keys, spos,
                                                                   rc2, offs, tot);
  k_rg_scan<<<dim3(1), dim3(1024), 0, s>>>(a.N, offs, tot, flags);
  return hipGetLastError();
}

hipError_t launch_radius_emit(const RadiusGraphArgs& a, char* ws, int max_candidates, int32_t* edge_index,
                              float* edge_vec, int32_t* edge_image, hipStream_t s) {
  if (a.N == 0) return hipSuccess;
  if (max_candidates < 0 || max_candidates > kRadiusMaxNeighbours) return hipErrorInvalidValue;
  const RadiusGraphLayout l = radius_graph_layout(a.N, a.G);
  int P = kWave;
  while (P < max_candidates) P <<= 1;
  const float rc2 = a.r_cut * a.r_cut;
  k_rg_emit<<<dim3(unsigned(a.N)), dim3(kWave), size_t(P) * 8, s>>>(
      a, reinterpret_cast<const GridParams*>(ws + l.params), reinterpret_cast<const int32_t*>(ws + l.keys),
      reinterpret_cast<const int32_t*>(ws + l.gid), reinterpret_cast<const int32_t*>(ws + l.cell_off), l.n_keys,
      reinterpret_cast<const float4*>(ws + l.spos), rc2, reinterpret_cast<const int32_t*>(ws + l.offs), P,
      edge_index, edge_vec, edge_image);
  return hipGetLastError();
}

}  // namespace tdn
