// Attention weights of the attention block that consumes the CP messages
// (Sec. 4.1, "Model Design": TDN keeps Equiformer's graph attention with MLP
// attention and replaces the tensor products inside it by the CP product
// with path-weight sharing).  For an edge e = (s, t):
//   q_e = [x[t]^(0), x[s]^(0), phi_e]               invariant inputs
//   a_e = LeakyReLU(q_e W1, 0.2) w2                 one logit per head
//   alpha_e[h] = softmax over the edges into t of a_e[h]
// q_e W1 splits into per-node parts, Pt[t] + Ps[s] + phi_e W1_phi, so the
// node parts are formed once per node (k_att_node) and the edge kernel
// (k_att_alpha, one wave per destination) adds them per edge.  The edge pass
// then weights each edge's message per head (launch_cp_edge_att).
#include "common.hpp"
#include "kernels.h"
#include "sh_device.hpp"

namespace tdn {

namespace {

constexpr int kAttMaxF = 64, kAttMaxH = 8, kAttMaxRadial = 16;
constexpr float kLeaky = 0.2f;
constexpr int kAttPer = 4;  // edges per lane whose logits stay in registers (segments up to 256 edges)

// Both projections of the degree-0 rows, Pt = X0 W1[0 .. C) and
// Ps = X0 W1[C .. 2C), tiled: a workgroup takes NB = 256 / FP nodes (FP =
// F rounded up to a power of two), one thread per (node, hidden unit), and
// the contraction over channels in chunks of 32 staged in LDS (the chunk's
// rows of both halves of W1 and of the nodes' degree-0 rows).
constexpr int kAttCk = 32;
__global__ __launch_bounds__(256) void k_att_node(int N, int d, int C, int F, int FP, const float* __restrict__ x,
                                                  const float* __restrict__ W1, float* __restrict__ Pt,
                                                  float* __restrict__ Ps) {
  __shared__ float sWt[kAttCk * kAttMaxF], sWs[kAttCk * kAttMaxF];
  __shared__ float sX[kAttCk * 256];  // [NB][kAttCk], NB <= 256
  const int NB = blockDim.x / FP;
  const int nl = threadIdx.x / FP, j = threadIdx.x - nl * FP;
  const int n = blockIdx.x * NB + nl;
  float pt = 0.f, ps = 0.f;
  for (int c0 = 0; c0 < C; c0 += kAttCk) {
    __syncthreads();  // the previous chunk consumed
    for (int i = threadIdx.x; i < kAttCk * F; i += blockDim.x) {
      const int c = i / F, jj = i - c * F;
      const bool ok = c0 + c < C;
      sWt[c * kAttMaxF + jj] = ok ? W1[(c0 + c) * F + jj] : 0.f;
      sWs[c * kAttMaxF + jj] = ok ? W1[(C + c0 + c) * F + jj] : 0.f;
    }
    for (int i = threadIdx.x; i < NB * kAttCk; i += blockDim.x) {
      const int r = i / kAttCk, c = i - r * kAttCk;
      const int nn = blockIdx.x * NB + r;
      sX[i] = (nn < N && c0 + c < C) ? x[size_t(nn) * d * C + c0 + c] : 0.f;
    }
    __syncthreads();
    if (j < F) {
#pragma unroll 8
      for (int c = 0; c < kAttCk; ++c) {
        const float v = sX[nl * kAttCk + c];
        pt = fmaf(v, sWt[c * kAttMaxF + j], pt);
        ps = fmaf(v, sWs[c * kAttMaxF + j], ps);
      }
    }
  }
  if (n < N && j < F) {
    Pt[size_t(n) * F + j] = pt;
    Ps[size_t(n) * F + j] = ps;
  }
}

// one wave per destination t: logits of its edges (one lane per edge, 64 at
// a time) into alpha_sorted, then per head the maximum and the sum of the
// exponentials by wave reductions in a fixed order, then the weights.  The
// radial rows of W1 and w2 are staged in LDS per workgroup; a lane reads its
// source's Ps row with 16-byte loads.
__global__ __launch_bounds__(4 * kWave) void k_att_alpha(int N, int C, int F, int H, int nr, float sigma,
                                                   const int32_t* __restrict__ offsets,
                                                   const int32_t* __restrict__ perm, const int32_t* __restrict__ src,
                                                   const float* __restrict__ edge_vec, const float* __restrict__ Pt,
                                                   const float* __restrict__ Ps, const float* __restrict__ W1,
                                                   const float* __restrict__ w2, float* __restrict__ alpha_sorted,
                                                   float* __restrict__ alpha_eid) {
  __shared__ float sWphi[kAttMaxRadial * kAttMaxF];
  __shared__ float sW2[kAttMaxF * kAttMaxH];
  __shared__ float sPt[4][kAttMaxF];  // each wave's destination row of Pt
  const float* Wphi = W1 + size_t(2 * C) * F;
  // zero-padded to kAttMaxRadial rows and kAttMaxH columns, so that the
  // per-unit loops below run to fixed bounds without guards (the padding
  // adds exact zeros)
  for (int i = threadIdx.x; i < kAttMaxRadial * F; i += blockDim.x) sWphi[i] = i < nr * F ? Wphi[i] : 0.f;
  for (int i = threadIdx.x; i < F * kAttMaxH; i += blockDim.x) {
    const int j = i / kAttMaxH, h = i - j * kAttMaxH;
    sW2[i] = h < H ? w2[j * H + h] : 0.f;
  }
  __syncthreads();
  const int lane = threadIdx.x & (kWave - 1);
  const int t = blockIdx.x * (blockDim.x / kWave) + int(threadIdx.x / kWave);
  if (t >= N) return;  // whole waves, after the only barrier
  const int e0 = offsets[t], e1 = offsets[t + 1];
  if (e0 >= e1) return;
  const int wv = threadIdx.x / kWave;
  if (lane < F) sPt[wv][lane] = Pt[size_t(t) * F + lane];
  // one wave writes and reads its row: its LDS operations run in order, and
  // the wave barrier keeps the compiler from moving the reads above the writes
  __builtin_amdgcn_wave_barrier();
  const bool vec4 = (F & 3) == 0;
  // the logits of sorted edge e into a[], its edge id into eid
  auto logit = [&](int e, float (&a)[kAttMaxH], int& eid) {
    eid = perm[e];
    const int s = src[eid];
    const float vx = edge_vec[3 * size_t(eid)], vy = edge_vec[3 * size_t(eid) + 1], vz = edge_vec[3 * size_t(eid) + 2];
    const float len = sqrtf(vx * vx + vy * vy + vz * vz);
    float phi[kAttMaxRadial];
#pragma unroll
    for (int q = 0; q < kAttMaxRadial; ++q) phi[q] = radial_phi(len, q, sigma);
#pragma unroll
    for (int h = 0; h < kAttMaxH; ++h) a[h] = 0.f;
    const float* pt = sPt[wv];
    const float* ps = Ps + size_t(s) * F;
    auto unit = [&](int j, float psj) {
      float hj = pt[j] + psj;
#pragma unroll
      for (int q = 0; q < kAttMaxRadial; ++q) hj = fmaf(phi[q], sWphi[q * F + j], hj);
      hj = hj > 0.f ? hj : kLeaky * hj;
#pragma unroll
      for (int h = 0; h < kAttMaxH; ++h) a[h] = fmaf(hj, sW2[j * kAttMaxH + h], a[h]);
    };
    if (vec4) {
      for (int j = 0; j < F; j += 4) {
        const float4 p4 = *reinterpret_cast<const float4*>(ps + j);
        unit(j, p4.x);
        unit(j + 1, p4.y);
        unit(j + 2, p4.z);
        unit(j + 3, p4.w);
      }
    } else {
      for (int j = 0; j < F; ++j) unit(j, ps[j]);
    }
  };
  auto wave_max = [&](float (&m)[kAttMaxH]) {
#pragma unroll
    for (int h = 0; h < kAttMaxH; ++h)
#pragma unroll
      for (int o = kWave / 2; o > 0; o >>= 1) m[h] = fmaxf(m[h], __shfl_xor(m[h], o));
  };
  auto wave_sum = [&](float (&m)[kAttMaxH]) {
#pragma unroll
    for (int h = 0; h < kAttMaxH; ++h)
#pragma unroll
      for (int o = kWave / 2; o > 0; o >>= 1) m[h] += __shfl_xor(m[h], o);
  };
  float mx[kAttMaxH], sm[kAttMaxH];
#pragma unroll
  for (int h = 0; h < kAttMaxH; ++h) {
    mx[h] = -INFINITY;
    sm[h] = 0.f;
  }
  if (e1 - e0 <= kAttPer * kWave) {
    // up to kAttPer edges per lane: the logits stay in registers
    float a[kAttPer][kAttMaxH];
    int eid[kAttPer];
#pragma unroll
    for (int u = 0; u < kAttPer; ++u) {
      const int e = e0 + lane + u * kWave;
      eid[u] = 0;
      if (e < e1) {
        logit(e, a[u], eid[u]);
#pragma unroll
        for (int h = 0; h < kAttMaxH; ++h) mx[h] = fmaxf(mx[h], a[u][h]);
      }
    }
    wave_max(mx);
#pragma unroll
    for (int u = 0; u < kAttPer; ++u)
      if (e0 + lane + u * kWave < e1)
#pragma unroll
        for (int h = 0; h < kAttMaxH; ++h) {
          a[u][h] = expf(a[u][h] - mx[h]);
          sm[h] += a[u][h];
        }
    wave_sum(sm);
#pragma unroll
    for (int u = 0; u < kAttPer; ++u) {
      const int e = e0 + lane + u * kWave;
      if (e < e1)
#pragma unroll
        for (int h = 0; h < kAttMaxH; ++h)
          if (h < H) {
            const float v = a[u][h] / sm[h];
            alpha_sorted[size_t(e) * H + h] = v;
            if (alpha_eid) alpha_eid[size_t(eid[u]) * H + h] = v;
          }
    }
    return;
  }
  // longer segments: the logits go through alpha_sorted
  for (int e = e0 + lane; e < e1; e += kWave) {
    float a[kAttMaxH];
    int eid;
    logit(e, a, eid);
#pragma unroll
    for (int h = 0; h < kAttMaxH; ++h)
      if (h < H) {
        alpha_sorted[size_t(e) * H + h] = a[h];
        mx[h] = fmaxf(mx[h], a[h]);
      }
  }
  wave_max(mx);
  for (int e = e0 + lane; e < e1; e += kWave)
#pragma unroll
    for (int h = 0; h < kAttMaxH; ++h)
      if (h < H) {
        const float v = expf(alpha_sorted[size_t(e) * H + h] - mx[h]);
        alpha_sorted[size_t(e) * H + h] = v;
        sm[h] += v;
      }
  wave_sum(sm);
  for (int e = e0 + lane; e < e1; e += kWave) {
    const int eid = alpha_eid ? perm[e] : 0;
#pragma unroll
    for (int h = 0; h < kAttMaxH; ++h)
      if (h < H) {
        const float v = alpha_sorted[size_t(e) * H + h] / sm[h];
        alpha_sorted[size_t(e) * H + h] = v;
        if (alpha_eid) alpha_eid[size_t(eid) * H + h] = v;
      }
  }
}

}  // namespace

hipError_t launch_att_node(int N, int d, int C, int F, const float* x, const float* W1, float* Pt, float* Ps,
                           hipStream_t s) {
  if (N == 0) return hipSuccess;
  if (F < 1 || F > kAttMaxF || !x || !W1 || !Pt || !Ps) return hipErrorInvalidValue;
  int FP = 1;
  while (FP < F) FP <<= 1;
  const int NB = 256 / FP;
  k_att_node<<<dim3((N + NB - 1) / NB), dim3(256), 0, s>>>(N, d, C, F, FP, x, W1, Pt, Ps);
  return hipGetLastError();
}

hipError_t launch_att_alpha(int N, int C, int F, int H, int n_radial, float sigma, const int32_t* offsets,
                            const int32_t* perm, const int32_t* src, const float* edge_vec, const float* Pt,
                            const float* Ps, const float* W1, const float* w2, float* alpha_sorted,
                            float* alpha_eid, hipStream_t s) {
  if (N == 0) return hipSuccess;
  if (F < 1 || F > kAttMaxF || H < 1 || H > kAttMaxH || n_radial < 1 || n_radial > kAttMaxRadial || !offsets ||
      !Pt || !Ps || !W1 || !w2)
    return hipErrorInvalidValue;
  k_att_alpha<<<dim3((N + 3) / 4), dim3(4 * kWave), 0, s>>>(N, C, F, H, n_radial, sigma, offsets, perm, src,
                                                            edge_vec, Pt, Ps, W1, w2, alpha_sorted, alpha_eid);
  return hipGetLastError();
}

}  // namespace tdn
