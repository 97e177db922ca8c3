// Batched decode, B <= 32 sequences with one token each (Section 5.2, Appendix C.1).
//
// With 32 tokens the gathered products become real dense contractions: every weight
// row fetched from HBM is used by all B tokens, so the work is done on the matrix
// cores (16x16x32 fp16 MFMA, fp32 accumulation) with the token batch as the N
// dimension, padded to NB = 16 or 32 with zero rows. The row sets are the union of
// the per-sequence sets (the union is what turns B sparse GEMVs into one sparse
// GEMM); each fetched row is read from HBM once per call.
//
//   k_union       union of B ascending index sets (LDS bitmap), its ranks, and
//                 per-row membership bits of the sequences.
//   k_ln_cast     x-hat = LN(x) (or x) as fp16 [NB][Kpad], zero padded.
//   k_mfma_rows   P[s][r][b] = sum_{k in split s} W[row(r)][k] x-hat[b][k]: gathered
//                 rows whose contraction index is contiguous in memory (fc1, Q/K/V,
//                 predictor factors). A workgroup stages one K-split of x-hat in LDS;
//                 each wavefront streams 16-row tiles straight into MFMA operands.
//   k_mfma_cols   P2[s][b][n] = sum_{u in split s} C[b][u] M[row(u)][n]: gathered rows
//                 contracted over the row index (fc2, out-projection). Row tiles are
//                 transposed through a per-wavefront LDS tile (XOR-swizzled, no bank
//                 conflicts) into the B operand.
//   finishers     sum the split partials in a fixed order and apply bias, ReLU,
//                 membership masks, cache writes and residuals.
#include <math.h>

#include "dv_internal.hpp"

namespace dv {

__device__ __forceinline__ f32x4 mfma16x16x32(f16x8 a, f16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// ------------------------------------------------------------------ union
// One workgroup. sets[b][0..k) ascending in [0, n). U receives the union in
// ascending order and *count its size; pos (optional) [n] the rank of i in U or -1;
// mask (optional) [>= |U|] bit b set iff U[u] is in set b.
template <int NT>
__global__ void __launch_bounds__(NT) k_union(const int32_t* __restrict__ sets, int B, int k, int n,
                                              int32_t* __restrict__ U, int32_t* __restrict__ count,
                                              int32_t* __restrict__ pos, uint32_t* __restrict__ mask) {
  extern __shared__ uint32_t usm[];
  const int nw = (n + 31) >> 5;
  uint32_t* bits = usm;
  int* off = reinterpret_cast<int*>(usm + nw);
  int* red = off + nw;
  const int tid = threadIdx.x;
  for (int w = tid; w < nw; w += NT) bits[w] = 0u;
  __syncthreads();
  const int tot = B * k;
  for (int e = tid; e < tot; e += NT) {
    const int i = min(max(sets[e], 0), n - 1);
    atomicOr(&bits[i >> 5], 1u << (i & 31));
  }
  __syncthreads();
  const int per = (nw + NT - 1) / NT;
  const int w0 = min(tid * per, nw), w1 = min(w0 + per, nw);
  int c = 0;
  for (int w = w0; w < w1; ++w) c += __popc(bits[w]);
  int total = 0;
  int base = block_excl_scan<NT>(c, red, &total);
  for (int w = w0; w < w1; ++w) {
    off[w] = base;
    uint32_t m = bits[w];
    while (m) {
      const int b = __ffs(m) - 1;
      U[base++] = w * 32 + b;
      m &= m - 1u;
    }
  }
  if (tid == 0) *count = total;
  __syncthreads();
  if (pos != nullptr) {
    for (int i = tid; i < n; i += NT) {
      const uint32_t m = bits[i >> 5];
      const uint32_t below = m & ((1u << (i & 31)) - 1u);
      pos[i] = ((m >> (i & 31)) & 1u) ? off[i >> 5] + __popc(below) : -1;
    }
  }
  if (mask != nullptr) {
    for (int u = tid; u < total; u += NT) mask[u] = 0u;
    __syncthreads();
    for (int e = tid; e < tot; e += NT) {
      const int i = min(max(sets[e], 0), n - 1);
      const uint32_t m = bits[i >> 5];
      const int r = off[i >> 5] + __popc(m & ((1u << (i & 31)) - 1u));
      atomicOr(&mask[r], 1u << (e / k));
    }
  }
}

hipError_t launch_union(const int32_t* sets, int B, int k, int n, int32_t* U, int32_t* count, int32_t* pos,
                        uint32_t* mask, hipStream_t st) {
  constexpr int NT = 1024;
  const int nw = (n + 31) >> 5;
  const size_t lds = (size_t)nw * 8 + (NT / 64 + 2) * sizeof(int);
  hipLaunchKernelGGL(k_union<NT>, dim3(1), dim3(NT), lds, st, sets, B, k, n, U, count, pos, mask);
  return hipGetLastError();
}

// --------------------------------------------------------------- x-hat cast
// X16[b][0..Kpad) = fp16(LN(x[b])) (g == NULL: x[b]) for b < B; zero for b >= B
// and for k >= d. One workgroup per row b of NB.
__global__ void __launch_bounds__(256) k_ln_cast(const float* __restrict__ x, int B, int d, int Kpad,
                                                 const float* __restrict__ g, const float* __restrict__ be,
                                                 float eps, _Float16* __restrict__ X16) {
  __shared__ float red[8];
  const int b = blockIdx.x;
  _Float16* o = X16 + (size_t)b * Kpad;
  if (b >= B) {
    for (int k = threadIdx.x; k < Kpad; k += 256) o[k] = (_Float16)0.f;
    return;
  }
  const float* xr = x + (size_t)b * d;
  float mean = 0.f, rstd = 1.f;
  if (g != nullptr) {
    float s = 0.f;
    for (int k = threadIdx.x; k < d; k += 256) s += xr[k];
    mean = block_sum<256>(s, red) / (float)d;
    float q = 0.f;
    for (int k = threadIdx.x; k < d; k += 256) {
      const float a = xr[k] - mean;
      q += a * a;
    }
    rstd = 1.0f / sqrtf(block_sum<256>(q, red) / (float)d + eps);
  }
  for (int k = threadIdx.x; k < Kpad; k += 256) {
    float v = 0.f;
    if (k < d) {
      v = xr[k];
      if (g != nullptr) v = (v - mean) * rstd * g[k] + (be ? be[k] : 0.f);
    }
    o[k] = (_Float16)v;
  }
}

hipError_t launch_ln_cast(const float* x, int B, int NB, int d, int Kpad, const float* g, const float* be, float eps,
                          _Float16* X16, hipStream_t st) {
  hipLaunchKernelGGL(k_ln_cast, dim3(NB), dim3(256), 0, st, x, B, d, Kpad, g, be, eps, X16);
  return hipGetLastError();
}

// ------------------------------------------------------------ k_mfma_rows
__device__ __forceinline__ int rows_count(const MrowsArgs& a) {
  if (a.mode == kRowsIdentity) return a.nrows;
  const int c = a.list_count ? min(*a.list_count, a.list_max) : a.list_max;
  return a.mode == kRowsList ? c : 3 * c * a.dh;
}

// Byte offset of row r's first element and its matrix (0..2).
__device__ __forceinline__ const char* rows_ptr(const MrowsArgs& a, int r, int nrows) {
  if (a.mode == kRowsIdentity) {
    return r < a.n0 ? static_cast<const char*>(a.W0) + (size_t)r * a.d * 2
                    : static_cast<const char*>(a.W1) + (size_t)(r - a.n0) * a.d * 2;
  }
  if (a.mode == kRowsList)
    return static_cast<const char*>(a.W0) + (size_t)min(max(a.list[r], 0), a.list_range - 1) * a.d * 2;
  const int per = nrows / 3;
  const int m = r / per;
  const int rem = r - m * per;
  const int p = rem / a.dh, t = rem - p * a.dh;
  const void* W = m == 0 ? a.W0 : (m == 1 ? a.W1 : a.W2);
  const int h = min(max(a.list[p], 0), a.list_range - 1);
  return static_cast<const char*>(W) + ((size_t)h * a.dh + t) * a.d * 2;
}

template <int NB, int U>
__device__ __forceinline__ void mr_load(u32x4 (&w)[U], const char* rp, bool rv, int kbyte0, int kvalid_bytes,
                                        int lg) {
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int kb = kbyte0 + u * 64 + lg * 16;
    w[u] = (rv && kb < kvalid_bytes) ? ld_stream(rp + kb) : u32x4{0u, 0u, 0u, 0u};
  }
}

template <int NB, int NW, int U>
__global__ void __launch_bounds__(NW * 64) k_mfma_rows(MrowsArgs a) {
  constexpr int NT = NW * 64;
  constexpr int NBT = NB / 16;
  extern __shared__ __attribute__((aligned(16))) _Float16 xs[];
  const int tid = threadIdx.x;
  const int s = blockIdx.x % a.S, g = blockIdx.x / a.S, G = gridDim.x / a.S;
  const int ldx = a.Ks + 8;                     // halves per staged row (16-byte pad)
  const int k0 = s * a.Ks;
  // ---- stage x-hat[:, k0 : k0 + Ks) (zero beyond Kpad)
  const int cpr = a.Ks >> 3;
  for (int i = tid; i < NB * cpr; i += NT) {
    const int b = i / cpr, c = i - b * cpr;
    const int k = k0 + 8 * c;
    const u32x4 v = k < a.Kpad ? ld_plain(a.X + (size_t)b * a.Kpad + k) : u32x4{0u, 0u, 0u, 0u};
    *reinterpret_cast<u32x4*>(xs + b * ldx + 8 * c) = v;
  }
  __syncthreads();

  const int n = rows_count(a);
  const int ntiles = (n + 15) >> 4;
  const int wave = tid >> 6, lane = tid & 63;
  const int lr = lane & 15, lg = lane >> 4;
  const int tstride = G * NW;
  int tile = g * NW + wave;
  if (tile >= ntiles) return;                    // no barrier follows
  const int nbat = a.Ks / (32 * U);              // batches of U k-steps per tile
  const int kvalid = min(a.Ks, a.d - k0) * 2;    // valid bytes of this split in a row
  const int kb0 = k0 * 2;

  auto row_of = [&](int t, const char** rp, bool* rv) {
    const int r = t * 16 + lr;
    *rv = r < n;
    *rp = rows_ptr(a, *rv ? r : 0, n) + kb0;
  };
  f32x4 acc[NBT];
#pragma unroll
  for (int j = 0; j < NBT; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const char* rp;
  bool rv;
  row_of(tile, &rp, &rv);
  int bi = 0;
  u32x4 wa[U];
  mr_load<NB, U>(wa, rp, rv, 0, kvalid, lg);
  for (;;) {
    int ntile = tile, nbi = bi + 1;
    const char* nrp = rp;
    bool nrv = rv;
    if (nbi == nbat) {
      nbi = 0;
      ntile = tile + tstride;
      if (ntile < ntiles) row_of(ntile, &nrp, &nrv);
    }
    const bool more = ntile < ntiles;
    u32x4 wb[U];
    if (more) mr_load<NB, U>(wb, nrp, nrv, nbi * U * 64, kvalid, lg);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int ks = bi * U + u;
      const f16x8 av = __builtin_bit_cast(f16x8, wa[u]);
#pragma unroll
      for (int j = 0; j < NBT; ++j) {
        const f16x8 bv = *reinterpret_cast<const f16x8*>(xs + (lr + 16 * j) * ldx + 32 * ks + 8 * lg);
        acc[j] = mfma16x16x32(av, bv, acc[j]);
      }
    }
    if (bi == nbat - 1) {
      // tile done: lane holds rows tile*16 + 4*lg + i, token columns lr + 16*j
#pragma unroll
      for (int j = 0; j < NBT; ++j) {
        const int b = lr + 16 * j;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = tile * 16 + 4 * lg + i;
          if (r < n) {
            if (a.out0 != nullptr) {
              if (b < a.B) {
                if (r < a.n0) a.out0[(size_t)b * a.ld0 + r] = acc[j][i];
                else a.out1[(size_t)b * a.ld1 + (r - a.n0)] = acc[j][i];
              }
            } else {
              a.P[((size_t)s * a.nrows_pad + r) * NB + b] = acc[j][i];
            }
          }
        }
        acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
    if (!more) break;
#pragma unroll
    for (int u = 0; u < U; ++u) wa[u] = wb[u];
    tile = ntile;
    bi = nbi;
    rp = nrp;
    rv = nrv;
  }
}

static int lds_budget() {
  static int cached = 0;
  if (cached == 0) {
    int dev = 0, v = 0;
    (void)hipGetDevice(&dev);
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess || v <= 0) v = 65536;
    cached = v;
  }
  return cached;
}

// K per split for k_mfma_rows: a multiple of 32 * kMrU halves whose staged slice of
// NB rows fits the LDS budget (at most 128 KB).
static constexpr int kMrU = 8;
void mrows_split(int Kpad, int NB, int* S, int* Ks) {
  const int budget = min(lds_budget(), 131072);
  const int unit = 32 * kMrU;
  int kmax = ((budget / (NB * 2) - 8) / unit) * unit;
  if (kmax < unit) kmax = unit;
  int s = (Kpad + kmax - 1) / kmax;
  int ks = (((Kpad + s - 1) / s) + unit - 1) / unit * unit;
  *S = s;
  *Ks = ks;
}

template <int NB>
static hipError_t launch_mrows_t(MrowsArgs a, hipStream_t st) {
  constexpr int NW = 8;
  const size_t lds = (size_t)NB * (a.Ks + 8) * 2;
  const auto kern = k_mfma_rows<NB, NW, kMrU>;
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)min(lds_budget(), 131072));
    attr = true;
  }
  const int G = max(1, device_cu_count() / a.S);
  hipLaunchKernelGGL(kern, dim3(G * a.S), dim3(NW * 64), lds, st, a);
  return hipGetLastError();
}

hipError_t launch_mrows(int NB, const MrowsArgs& a, hipStream_t st) {
  return NB <= 16 ? launch_mrows_t<16>(a, st) : launch_mrows_t<32>(a, st);
}

// ------------------------------------------------------------ k_mfma_cols
// Rows of the contraction: M[list[u]] (dh == 0) or M[list[u / dh] * dh + u % dh].
__device__ __forceinline__ int cols_count(const McolsArgs& a) {
  const int c = a.list_count ? min(*a.list_count, a.list_max) : a.list_max;
  return a.dh > 0 ? c * a.dh : c;
}
__device__ __forceinline__ size_t cols_row(const McolsArgs& a, int u) {
  if (a.dh == 0) return (size_t)min(max(a.list[u], 0), a.list_range - 1);
  const int p = u / a.dh;
  return (size_t)min(max(a.list[p], 0), a.list_range - 1) * a.dh + (u - p * a.dh);
}

// Wavefront tile in LDS: 32 rows x 64 columns fp16, 16-byte chunk c of row r stored at
// chunk c ^ (2 * ((r >> 3) & 3)) so that both the row-wise 16-byte writes and the
// column-wise 2-byte reads of the transpose are free of bank conflicts.
template <int NB, int U>
struct ColsStep {
  u32x4 w[U][4];        // weights: rows (lane >> 3) + 8*i, 16-byte chunk lane & 7
  u32x4 h[U][NB / 16];  // coefficients: token lr + 16*j, rows 8*lg .. 8*lg + 7
};

template <int NB, int U>
__device__ __forceinline__ void mc_load(ColsStep<NB, U>& st, const McolsArgs& a, const char* Mb, int q0, int qend,
                                        int qstride, int uend, bool col_on, int lane) {
  const int lr = lane & 15, lg = lane >> 4;
  const size_t rowb = (size_t)a.d * 2;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int q = q0 + u * qstride;
    const bool on = q < qend;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 32 * q + (lane >> 3) + 8 * i;
      st.w[u][i] = (on && col_on && row < uend) ? ld_stream(Mb + cols_row(a, row) * rowb) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int j = 0; j < NB / 16; ++j)
      st.h[u][j] = on ? ld_plain(a.C + (size_t)(lr + 16 * j) * a.ldc + 32 * q + 8 * lg) : u32x4{0u, 0u, 0u, 0u};
  }
}

template <int NB, int NW, int U>
__global__ void __launch_bounds__(NW * 64) k_mfma_cols(McolsArgs a) {
  constexpr int NBT = NB / 16;
  extern __shared__ __attribute__((aligned(16))) _Float16 csm[];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int lr = lane & 15, lg = lane >> 4;
  _Float16* tile = csm + wave * (32 * 64);
  float* red = reinterpret_cast<float*>(csm + NW * 32 * 64);     // [NW][NB][64]
  const int n0 = blockIdx.x * 64;
  const int s = blockIdx.y;
  const int n = cols_count(a);
  const int us = ((n + a.S - 1) / a.S + 31) & ~31;
  const int ubeg = s * us, uend = min(n, ubeg + us);
  const int qbeg = ubeg >> 5, qend = (uend + 31) >> 5;
  const bool col_on = n0 + 8 * (lane & 7) < a.d;
  const char* Mb = static_cast<const char*>(a.M) + (size_t)(col_on ? n0 + 8 * (lane & 7) : 0) * 2;

  f32x4 acc[NBT][4];
#pragma unroll
  for (int j = 0; j < NBT; ++j)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[j][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int qstride = NW;
  int q = qbeg + wave;
  ColsStep<NB, U> cur;
  mc_load<NB, U>(cur, a, Mb, q, qend, qstride, uend, col_on, lane);
  for (; q < qend; q += qstride * U) {
    ColsStep<NB, U> nxt;
    const bool more = q + qstride * U < qend;
    if (more) mc_load<NB, U>(nxt, a, Mb, q + qstride * U, qend, qstride, uend, col_on, lane);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (q + u * qstride >= qend) break;
      // row-wise write of the 32 x 64 tile
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = (lane >> 3) + 8 * i;
        const int c = (lane & 7) ^ (2 * i);
        *reinterpret_cast<u32x4*>(tile + r * 64 + c * 8) = cur.w[u][i];
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      f16x8 hv[NBT];
#pragma unroll
      for (int j = 0; j < NBT; ++j) hv[j] = __builtin_bit_cast(f16x8, cur.h[u][j]);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        // column-wise read: token-major B operand, rows 8*lg .. 8*lg + 7 of column 16t + lr
        const int nl = 16 * t + lr;
        const int pc = (nl >> 3) ^ (2 * lg);
        const _Float16* src = tile + (8 * lg) * 64 + pc * 8 + (nl & 7);
        f16x8 bv;
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) bv[jj] = src[jj * 64];
#pragma unroll
        for (int j = 0; j < NBT; ++j) acc[j][t] = mfma16x16x32(hv[j], bv, acc[j][t]);
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    if (!more) break;
    cur = nxt;
  }
  // ---- reduce the wavefronts' partials in a fixed order
#pragma unroll
  for (int j = 0; j < NBT; ++j)
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[(wave * NB + 16 * j + 4 * lg + i) * 64 + 16 * t + lr] = acc[j][t][i];
  __syncthreads();
  for (int e = tid; e < NB * 64; e += NW * 64) {
    const int b = e >> 6, c = e & 63;
    if (b < a.B && n0 + c < a.d) {
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) v += red[(w * NB + b) * 64 + c];
      a.P[((size_t)s * a.B + b) * a.d + n0 + c] = v;
    }
  }
}

static constexpr int kMcNW = 4, kMcU = 2;

int mcols_split(int d, int nmax) {
  const int tiles = (d + 63) / 64;
  const int target = 2 * device_cu_count();
  int s = (target + tiles - 1) / tiles;
  const int q = (nmax + 31) / 32;                  // k-steps available
  s = max(1, min(s, max(1, q / (2 * kMcNW))));
  return min(s, 16);
}

template <int NB>
static hipError_t launch_mcols_t(const McolsArgs& a, hipStream_t st) {
  const size_t lds = (size_t)kMcNW * 32 * 64 * 2 + (size_t)kMcNW * NB * 64 * 4;
  dim3 grid((a.d + 63) / 64, a.S);
  hipLaunchKernelGGL((k_mfma_cols<NB, kMcNW, kMcU>), grid, dim3(kMcNW * 64), lds, st, a);
  return hipGetLastError();
}

hipError_t launch_mcols(int NB, const McolsArgs& a, hipStream_t st) {
  return NB <= 16 ? launch_mcols_t<16>(a, st) : launch_mcols_t<32>(a, st);
}

// --------------------------------------------------------------- finishers
// fc1: C[b][u] = fp16(ReLU(sum_s P[s][u][b] + b1[list[u]])) for b < B and u < n (and,
// with a mask, only where bit b of mask[u] is set); zero elsewhere up to a multiple
// of 64 rows. One workgroup per 64 rows.
template <int NB>
__global__ void __launch_bounds__(256) k_fc1_finish(Fc1FinishArgs a) {
  __shared__ float t[64][NB + 1];
  const int n = a.list_count ? min(*a.list_count, a.list_max) : a.list_max;
  const int u0 = blockIdx.x * 64;
  if (u0 >= ((n + 63) & ~63)) return;
  for (int e = threadIdx.x; e < 64 * NB; e += 256) {
    const int ul = e / NB, b = e - ul * NB;
    const int u = u0 + ul;
    float v = 0.f;
    if (u < n && b < a.B) {
      for (int s = 0; s < a.S; ++s) v += a.P[((size_t)s * a.nrows_pad + u) * NB + b];
      if (a.b1) v += a.b1[min(max(a.list[u], 0), a.list_range - 1)];
      v = v > 0.f ? v : 0.f;
      if (a.mask && !((a.mask[u] >> b) & 1u)) v = 0.f;
    }
    t[ul][b] = v;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < 64 * NB; e += 256) {
    const int b = e >> 6, ul = e & 63;
    a.C[(size_t)b * a.ldc + u0 + ul] = (_Float16)t[ul][b];
  }
}

hipError_t launch_fc1_finish(int NB, const Fc1FinishArgs& a, hipStream_t st) {
  const int blocks = max(1, (a.list_max + 63) / 64);
  if (NB <= 16)
    hipLaunchKernelGGL(k_fc1_finish<16>, dim3(blocks), dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(k_fc1_finish<32>, dim3(blocks), dim3(256), 0, st, a);
  return hipGetLastError();
}

// Sum of k_mfma_cols partials: out[b][c] = sum_s P2[s][b][c] + bias[c] + resid[b][c].
__global__ void __launch_bounds__(256) k_cols_finish(ColsFinishArgs a) {
  const long total = (long)a.B * a.d;
  for (long e = (long)blockIdx.x * 256 + threadIdx.x; e < total; e += (long)gridDim.x * 256) {
    const int c = (int)(e % a.d);
    float v = 0.f;
    for (int s = 0; s < a.S; ++s) v += a.P[(size_t)s * total + e];
    if (a.bias) v += a.bias[c];
    if (a.resid) v += a.resid[e];
    a.out[e] = v;
  }
}

hipError_t launch_cols_finish(const ColsFinishArgs& a, hipStream_t st) {
  const long total = (long)a.B * a.d;
  const long want = (total + 255) / 256, cap = 4L * device_cu_count();
  const int blocks = (int)(want < cap ? want : cap);
  hipLaunchKernelGGL(k_cols_finish, dim3(max(1, blocks)), dim3(256), 0, st, a);
  return hipGetLastError();
}

// Predictor hidden layer: C[b][j] = fp16(sum_s P[s][j][b]) for j < r, b < B (zero
// padding to ldc columns and NB rows).
template <int NB>
__global__ void __launch_bounds__(256) k_sum_cast(const float* __restrict__ P, int S, int nrows_pad, int row0,
                                                  int r, int B, _Float16* __restrict__ C, int ldc) {
  const int total = NB * ldc;
  for (int e = blockIdx.x * 256 + threadIdx.x; e < total; e += gridDim.x * 256) {
    const int b = e / ldc, j = e - b * ldc;
    float v = 0.f;
    if (b < B && j < r)
      for (int s = 0; s < S; ++s) v += P[((size_t)s * nrows_pad + row0 + j) * NB + b];
    C[e] = (_Float16)v;
  }
}

hipError_t launch_sum_cast(int NB, const float* P, int S, int nrows_pad, int row0, int r, int B, _Float16* C, int ldc,
                           hipStream_t st) {
  const int blocks = min((NB * ldc + 255) / 256, 4 * device_cu_count());
  if (NB <= 16)
    hipLaunchKernelGGL(k_sum_cast<16>, dim3(blocks), dim3(256), 0, st, P, S, nrows_pad, row0, r, B, C, ldc);
  else
    hipLaunchKernelGGL(k_sum_cast<32>, dim3(blocks), dim3(256), 0, st, P, S, nrows_pad, row0, r, B, C, ldc);
  return hipGetLastError();
}

// Q/K/V of the batch: for sequence b and its j-th selected head h (union rank p),
// value of projection m at t = sum_s P[s][(m*nu + p)*dh + t][b] + bias; q goes to
// q[b][j][t], k and v to the cache at row pos[b] of head h (round to nearest even).
template <int NB, typename KT>
__global__ void __launch_bounds__(256) k_qkv_finish(QkvFinishArgs a) {
  const int j = blockIdx.x, b = blockIdx.y;
  const int h = min(max(a.heads[(size_t)b * a.n_heads + j], 0), a.H - 1);
  const int p = a.hpos[h];
  const int nu = *a.hcount;
  const int pos = a.posb[b];
  if (p < 0 || p >= nu) return;
  for (int e = threadIdx.x; e < 3 * a.dh; e += 256) {
    const int m = e / a.dh, t = e - m * a.dh;
    const int r = (m * nu + p) * a.dh + t;
    float v = 0.f;
    for (int s = 0; s < a.S; ++s) v += a.P[((size_t)s * a.nrows_pad + r) * NB + b];
    const float* bias = m == 0 ? a.bq : (m == 1 ? a.bk : a.bv);
    if (bias) v += bias[(size_t)h * a.dh + t];
    if (m == 0) {
      a.q[((size_t)b * a.n_heads + j) * a.dh + t] = v;
    } else {
      KT* Cc = static_cast<KT*>(m == 1 ? a.K : a.V);
      Cc[(((size_t)b * a.H + h) * a.cap + pos) * a.dh + t] = (KT)v;
    }
  }
}

hipError_t launch_qkv_finish(int NB, int kvtype, const QkvFinishArgs& a, hipStream_t st) {
  dim3 grid(a.n_heads, a.B);
  if (NB <= 16) {
    if (kvtype == DV_F16) hipLaunchKernelGGL((k_qkv_finish<16, _Float16>), grid, dim3(256), 0, st, a);
    else hipLaunchKernelGGL((k_qkv_finish<16, float>), grid, dim3(256), 0, st, a);
  } else {
    if (kvtype == DV_F16) hipLaunchKernelGGL((k_qkv_finish<32, _Float16>), grid, dim3(256), 0, st, a);
    else hipLaunchKernelGGL((k_qkv_finish<32, float>), grid, dim3(256), 0, st, a);
  }
  return hipGetLastError();
}

// Attention outputs as out-projection coefficients: C[b][p*dh + t] = H_h(x_b)[t] for
// the union head h = list[p] if h is in sequence b's set (combining its split-KV
// partials), else 0; rows up to ldc are covered (zero beyond the union).
__global__ void __launch_bounds__(256) k_attn_finish(AttnFinishArgs a) {
  __shared__ float fac[kAttnMaxSplit];
  __shared__ int jsel;
  const int p = blockIdx.x, b = blockIdx.y;
  const int nu = *a.hcount;
  const int r0 = p * a.dh;
  if (r0 >= a.ldc) return;
  _Float16* o = a.C + (size_t)b * a.ldc + r0;
  const int rows = min(a.dh, a.ldc - r0);
  if (threadIdx.x == 0) {
    int jj = -1;
    if (p < nu && b < a.B) {
      const int h = a.list[p];   // union entries are in range by construction
      const int32_t* hs = a.heads + (size_t)b * a.n_heads;
      int lo = 0, hi = a.n_heads - 1;
      while (lo <= hi) {
        const int mid = (lo + hi) >> 1;
        if (hs[mid] == h) { jj = mid; break; }
        if (hs[mid] < h) lo = mid + 1; else hi = mid - 1;
      }
    }
    jsel = jj;
    if (jj >= 0) {
      const float* P = a.part + ((size_t)b * a.n_heads + jj) * a.n_split * (a.dh + 2);
      float M = -INFINITY;
      for (int c = 0; c < a.n_split; ++c) M = fmaxf(M, P[(size_t)c * (a.dh + 2)]);
      float L = 0.f;
      for (int c = 0; c < a.n_split; ++c) {
        const float m = P[(size_t)c * (a.dh + 2)];
        const float f = m == -INFINITY ? 0.f : __expf(m - M);
        fac[c] = f;
        L += P[(size_t)c * (a.dh + 2) + 1] * f;
      }
      for (int c = 0; c < a.n_split; ++c) fac[c] /= L;
    }
  }
  __syncthreads();
  const int jj = jsel;
  for (int t = threadIdx.x; t < rows; t += 256) {
    float v = 0.f;
    if (jj >= 0 && t < a.dh) {
      const float* P = a.part + ((size_t)b * a.n_heads + jj) * a.n_split * (a.dh + 2) + 2 + t;
      for (int c = 0; c < a.n_split; ++c) v += P[(size_t)c * (a.dh + 2)] * fac[c];
    }
    o[t] = (_Float16)v;
  }
}

hipError_t launch_attn_finish(int NB, const AttnFinishArgs& a, hipStream_t st) {
  dim3 grid((a.ldc + a.dh - 1) / a.dh, NB);
  hipLaunchKernelGGL(k_attn_finish, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace dv
