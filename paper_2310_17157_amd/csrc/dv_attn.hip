// Sparsified multi-head attention (Eq. (2), Section 2.3) at decode time, with the
// KV-cache rule of Section 4.2 (keys and values are computed and stored only for the
// selected heads).
//
//   k_qkv   gathered row-dots: for every selected head i, the dh rows of W^Q_i, W^K_i
//           and W^V_i (contiguous row blocks) against the staged x-hat; q goes to the
//           workspace, k and v to cache row pos. Optionally selects the head set
//           itself from the head predictor's scores (ranked in every workgroup).
//   k_attn  split-KV decode attention: one workgroup per (selected head, position
//           chunk) computes the chunk's max logit, sum of exponentials and
//           unnormalised value sum; the out-projection kernel combines the chunks.
#include <math.h>

#include "dv_internal.hpp"
#include "dv_select.hpp"   // wg_topk_small

namespace dv {

template <typename T, typename KT, int NW, int U>
__global__ void __launch_bounds__(NW * 64) k_qkv(QkvArgs a) {
  extern __shared__ float smem[];
  constexpr int NT = NW * 64;
  float* xs = smem;
  float* red = smem + a.d;
  int32_t* hset = reinterpret_cast<int32_t*>(red + NW);
  int* tmp = hset + a.n_heads;                                  // H ints
  uint32_t* hkeys = reinterpret_cast<uint32_t*>(tmp + a.H);     // H keys
  if (a.heads_in != nullptr) {
    for (int i = threadIdx.x; i < a.n_heads; i += NT) hset[i] = min(max(a.heads_in[i], 0), a.H - 1);
    __syncthreads();
  } else {
    wg_topk_small<NT>(a.head_scores, a.H, a.n_heads, hkeys, tmp, hset);
  }
  if (blockIdx.x == 0) {
    for (int i = threadIdx.x; i < a.n_heads; i += NT) {
      a.heads_ws[i] = hset[i];
      if (a.heads_out) a.heads_out[i] = hset[i];
    }
  }
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int per_mat = a.n_heads * a.dh;
  const int nrows = 3 * per_mat;
  const int nblk = gridDim.x;
  struct RowRef { const T* p; int m, rem, head, t; };
  auto row_ref = [&](int row) {
    RowRef r;
    r.m = row / per_mat;
    r.rem = row - r.m * per_mat;
    const int j = r.rem / a.dh;
    r.t = r.rem - j * a.dh;
    r.head = hset[j];
    const void* W = r.m == 0 ? a.Wq : (r.m == 1 ? a.Wk : a.Wv);
    r.p = static_cast<const T*>(W) + ((size_t)r.head * a.dh + r.t) * a.d;
    return r;
  };
  // Issue the first row's loads before the layer-norm prologue.
  u32x4 pf[U];
  {
    const int row0 = blockIdx.x * NW + wave;
    if (row0 < nrows) row_prefetch<T, U, 1>(row_ref(row0).p, a.d, lane, 0, pf);
  }
  stage_x<T, NT>(a.x, a.d, a.g, a.be, a.eps, xs, red);

  bool first = true;
  for (int row = blockIdx.x * NW + wave; row < nrows; row += nblk * NW) {
    const RowRef r = row_ref(row);
    const int m = r.m, rem = r.rem, head = r.head, t = r.t;
    const size_t wrow = (size_t)head * a.dh + t;
    float v = first ? wave_rowdot_pf<T, U, 1>(r.p, xs, a.d, lane, 0, pf) : wave_rowdot<T, U, 1>(r.p, xs, a.d, lane, 0);
    first = false;
    if (lane == 0) {
      const float* bias = m == 0 ? a.bq : (m == 1 ? a.bk : a.bv);
      if (bias) v += bias[wrow];
      if (m == 0) {
        a.q[rem] = v;
      } else {
        KT* C = static_cast<KT*>(m == 1 ? a.K : a.V);
        C[((size_t)head * a.cap + a.pos) * a.dh + t] = (KT)v;
      }
    }
  }
}

template <typename T, typename KT>
static hipError_t launch_qkv_t(const QkvArgs& a, hipStream_t st) {
  constexpr int NW = 8, U = 8;
  const int nrows = 3 * a.n_heads * a.dh;
  const int cus = device_cu_count();
  // Every row is one wavefront task; cap the grid at a few resident workgroups per CU.
  int blocks = min((nrows + NW - 1) / NW, 2 * cus);
  blocks = max(blocks, 1);
  size_t lds = (size_t)(a.d + NW) * sizeof(float) + (size_t)(a.n_heads + 2 * a.H + 4) * sizeof(int32_t);
  hipLaunchKernelGGL((k_qkv<T, KT, NW, U>), dim3(blocks), dim3(NW * 64), lds, st, a);
  return hipGetLastError();
}

hipError_t launch_qkv(int wtype, int kvtype, const QkvArgs& a, hipStream_t st) {
  if (wtype == DV_F16)
    return kvtype == DV_F16 ? launch_qkv_t<_Float16, _Float16>(a, st) : launch_qkv_t<_Float16, float>(a, st);
  return kvtype == DV_F16 ? launch_qkv_t<float, _Float16>(a, st) : launch_qkv_t<float, float>(a, st);
}

// ------------------------------------------------------------ attention
// LPP lanes hold one cache row (dh elements, 16 bytes per lane); a wavefront covers
// 64 / LPP positions per step and NSTEP steps; NW wavefronts per workgroup.
template <typename KT, int LPP, int NSTEP>
__global__ void __launch_bounds__(256) k_attn(AttnArgs a) {
  constexpr int NW = 4;
  constexpr int E = Chunk<KT>::E;
  constexpr int PPW = 64 / LPP;
  __shared__ float sm_m[NW], sm_l[NW];
  __shared__ float sm_o[NW][256];
  const int j = blockIdx.y, c = blockIdx.x;
  const int head = min(max(a.heads[j], 0), a.H - 1);
  const int t0 = c * a.chunk;
  const int tend = min(t0 + a.chunk, a.pos + 1);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int grp = lane / LPP, gl = lane % LPP;
  const int nchr = a.dh / E;
  const bool lane_on = gl < nchr;
  float qv[E];
#pragma unroll
  for (int e = 0; e < E; ++e) qv[e] = lane_on ? a.q[(size_t)j * a.dh + gl * E + e] : 0.f;
  const size_t rowb = (size_t)a.dh * sizeof(KT);
  const char* Kb = static_cast<const char*>(a.K) + (size_t)head * a.cap * rowb + (size_t)gl * 16;
  const char* Vb = static_cast<const char*>(a.V) + (size_t)head * a.cap * rowb + (size_t)gl * 16;

  u32x4 kw[NSTEP];
#pragma unroll
  for (int s = 0; s < NSTEP; ++s) {
    const int t = t0 + (s * NW + wave) * PPW + grp;
    kw[s] = (t < tend && lane_on) ? ld_plain(Kb + (size_t)t * rowb) : u32x4{0u, 0u, 0u, 0u};
  }
  float sc[NSTEP];
  float m = -INFINITY;
#pragma unroll
  for (int s = 0; s < NSTEP; ++s) {
    float kv[E];
    unpack<KT>(kw[s], kv);
    float p = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) p = fmaf(qv[e], kv[e], p);
#pragma unroll
    for (int o = LPP / 2; o > 0; o >>= 1) p += __shfl_xor(p, o, kWave);
    const int t = t0 + (s * NW + wave) * PPW + grp;
    sc[s] = t < tend ? p * a.scale : -INFINITY;
    m = fmaxf(m, sc[s]);
  }
#pragma unroll
  for (int o = LPP; o < 64; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, kWave));

  u32x4 vw[NSTEP];
#pragma unroll
  for (int s = 0; s < NSTEP; ++s) {
    const int t = t0 + (s * NW + wave) * PPW + grp;
    vw[s] = (t < tend && lane_on) ? ld_plain(Vb + (size_t)t * rowb) : u32x4{0u, 0u, 0u, 0u};
  }
  float l = 0.f;
  float o[E];
#pragma unroll
  for (int e = 0; e < E; ++e) o[e] = 0.f;
#pragma unroll
  for (int s = 0; s < NSTEP; ++s) {
    const float p = sc[s] == -INFINITY ? 0.f : __expf(sc[s] - m);
    l += p;
    float vv[E];
    unpack<KT>(vw[s], vv);
#pragma unroll
    for (int e = 0; e < E; ++e) o[e] = fmaf(p, vv[e], o[e]);
  }
#pragma unroll
  for (int off = LPP; off < 64; off <<= 1) {
    l += __shfl_xor(l, off, kWave);
#pragma unroll
    for (int e = 0; e < E; ++e) o[e] += __shfl_xor(o[e], off, kWave);
  }
  if (lane == 0) {
    sm_m[wave] = m;
    sm_l[wave] = l;
  }
  if (grp == 0 && lane_on) {
#pragma unroll
    for (int e = 0; e < E; ++e) sm_o[wave][gl * E + e] = o[e];
  }
  __syncthreads();
  float M = -INFINITY;
#pragma unroll
  for (int w = 0; w < NW; ++w) M = fmaxf(M, sm_m[w]);
  float* out = a.part + ((size_t)j * a.n_split + c) * (a.dh + 2);
  if (M == -INFINITY) {
    for (int t = threadIdx.x; t < a.dh + 2; t += 256) out[t] = t == 0 ? -INFINITY : 0.f;
    return;
  }
  float f[NW];
  float L = 0.f;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    f[w] = sm_m[w] == -INFINITY ? 0.f : __expf(sm_m[w] - M);
    L += sm_l[w] * f[w];
  }
  for (int t = threadIdx.x; t < a.dh; t += 256) {
    float acc = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) acc += sm_o[w][t] * f[w];
    out[2 + t] = acc;
  }
  if (threadIdx.x == 0) {
    out[0] = M;
    out[1] = L;
  }
}

int attn_chunk(int n_heads, int attended, int dh, int kvtype) {
  // Positions per workgroup: a multiple of the 4 wavefronts x positions per step, at
  // most 16 steps per wavefront; prefer long chunks (fewer partials) while keeping
  // about 2 workgroups per CU busy.
  const int nchr = dh * elem_bytes(kvtype) / 16;
  const int lpp = nchr <= 16 ? 16 : (nchr <= 32 ? 32 : 64);
  const int ppw = 64 / lpp;
  const int cmax = 16 * 4 * ppw, cmin = 4 * 4 * ppw;
  const int target = 2 * device_cu_count();
  for (int ch = cmax; ch > cmin; ch >>= 1)
    if ((long)n_heads * ((attended + ch - 1) / ch) >= target) return ch;
  return cmin;
}

template <typename KT, int LPP>
static hipError_t launch_attn_l(const AttnArgs& a, hipStream_t st) {
  constexpr int PPW = 64 / LPP;
  const int nstep = a.chunk / (4 * PPW);
  dim3 grid(a.n_split, a.n_heads);
  switch (nstep) {
    case 4: hipLaunchKernelGGL((k_attn<KT, LPP, 4>), grid, dim3(256), 0, st, a); break;
    case 8: hipLaunchKernelGGL((k_attn<KT, LPP, 8>), grid, dim3(256), 0, st, a); break;
    case 16: hipLaunchKernelGGL((k_attn<KT, LPP, 16>), grid, dim3(256), 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename KT>
static hipError_t launch_attn_t(const AttnArgs& a, hipStream_t st) {
  const int nchr = a.dh * (int)sizeof(KT) / 16;
  if (nchr <= 16) return launch_attn_l<KT, 16>(a, st);
  if (nchr <= 32) return launch_attn_l<KT, 32>(a, st);
  return launch_attn_l<KT, 64>(a, st);
}

hipError_t launch_attn(int kvtype, const AttnArgs& a, hipStream_t st) {
  return kvtype == DV_F16 ? launch_attn_t<_Float16>(a, st) : launch_attn_t<float>(a, st);
}

}  // namespace dv
