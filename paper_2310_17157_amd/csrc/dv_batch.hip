// Batched decode, B <= 32 sequences with one token each (Section 5.2, Appendix C.1).
//
// With 32 tokens the gathered products become real dense contractions: every weight
// row fetched from HBM is used by all B tokens, so the work is done on the matrix
// cores (16x16x32 fp16 MFMA, fp32 accumulation) with the token batch as the N
// dimension, padded to NB = 16 or 32 with zero rows. The row sets are the union of
// the per-sequence sets (the union is what turns B sparse GEMVs into one sparse
// GEMM); each fetched row is read from HBM once per call.
//
//   k_union_*     union of B ascending index sets (chunked bitmaps, then ranks), and
//                 per-row membership bits of the sequences.
//   k_ln_cast     x-hat = LN(x) (or x) as fp16 [NB][Kpad], zero padded.
//   k_mfma_rows   P[s][r][b] = sum_{k in split s} W[row(r)][k] x-hat[b][k]: gathered
//                 rows whose contraction index is contiguous in memory (fc1, Q/K/V,
//                 predictor factors). A workgroup stages one K-split of x-hat in LDS;
//                 each wavefront streams 16-row tiles straight into MFMA operands.
//   k_mfma_cols   P2[s][b][n] = sum_{u in split s} C(b, u) M[row(u)][n]: gathered rows
//                 contracted over the row index (fc2, out-projection). Row tiles are
//                 written to a per-wavefront LDS tile (XOR-swizzled) and read back
//                 column-wise with the LDS transpose read into the B operand.
//   finishers     sum the split partials in a fixed order and apply bias, ReLU,
//                 membership masks, cache writes and residuals.
#include <math.h>

#include "dv_internal.hpp"

namespace dv {

__device__ __forceinline__ f32x4 mfma16x16x32(f16x8 a, f16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

typedef short v4s_t __attribute__((ext_vector_type(4)));
typedef _Float16 f16x4_t __attribute__((ext_vector_type(4)));

// gfx950 LDS transpose read of four 16-bit elements (p: 8-byte aligned LDS address).
__device__ __forceinline__ v4s_t ds_read_tr16(const _Float16* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (v4s_t __attribute__((address_space(3)))*)(const_cast<_Float16*>(p)));
}

// ------------------------------------------------------------------ union
// Union of B ascending sets sets[b][0..k) in [0, n) in one launch, one workgroup per
// chunk of kUnionChunk indices. Every workgroup reads all B * k entries (they stay
// in L2) and marks a byte per index below its chunk's end in LDS (plain stores, so
// entries shared by many sets do not contend); the members below the chunk give
// its offset, the marks inside it the ranks. U[offset + rank] = the members in
// ascending order, *count = their number (last chunk), and optionally
// mask[offset + rank] = the member's sets as bits (bit b: set b holds it), gathered
// by LDS atomics on one word per index of the chunk.
constexpr int kUnionChunk = 2048;
constexpr int kUnionNT = 1024;
static_assert(kUnionChunk == 2 * kUnionNT, "two indices of the chunk per thread");

// Calls fn(e, v) for every entry e of sets[0..total) with value v. The entries are
// read as aligned int4 with all of a thread's loads in flight (one round trip for up
// to PER * 4 * kUnionNT entries; rounds of loads past the end are not issued). sets
// need only be 4-byte aligned: the quads start at its 16-byte block, so the first and
// the last quad may reach up to 12 bytes outside [sets, sets + total). Those bytes share
// an aligned 16-byte block with an entry, and such a block never crosses a page (GPU
// pages are at least 4 KB), so they are readable; their values are skipped.
template <class Fn>
__device__ __forceinline__ void union_scan(const int32_t* __restrict__ sets, int total, Fn fn) {
  constexpr int PER = 16;
  if (total <= 0) return;
  const int shift = (int)(((uintptr_t)sets & 15u) >> 2);
  const int4* base = reinterpret_cast<const int4*>((uintptr_t)sets & ~(uintptr_t)15u);
  const int n4 = (total + shift + 3) >> 2;
  for (int q0 = 0; q0 < n4; q0 += PER * kUnionNT) {
    const int nu = min(PER, (n4 - q0 + kUnionNT - 1) / kUnionNT);   // rounds of quads left (workgroup-uniform)
    int4 v[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u)
      v[u] = u < nu ? base[min(q0 + u * kUnionNT + (int)threadIdx.x, n4 - 1)] : make_int4(0, 0, 0, 0);
#pragma unroll
    for (int u = 0; u < PER; ++u) {   // quads of rounds not loaded have e >= total
      const int e = 4 * (q0 + u * kUnionNT + (int)threadIdx.x) - shift;
      if (e + 0 >= 0 && e + 0 < total) fn(e + 0, v[u].x);
      if (e + 1 >= 0 && e + 1 < total) fn(e + 1, v[u].y);
      if (e + 2 >= 0 && e + 2 < total) fn(e + 2, v[u].z);
      if (e + 3 >= 0 && e + 3 < total) fn(e + 3, v[u].w);
    }
  }
}

// Sum of four 0/1 bytes.
__device__ __forceinline__ int byte_flags(uint32_t w) { return (int)((w * 0x01010101u) >> 24); }

// Chunk c of nc; ush: dynamic LDS, marks [round_up(n, 16)] bytes, then (mask only)
// kUnionChunk words.
template <bool MASK>
__device__ __forceinline__ void union_chunk(const int32_t* __restrict__ sets, int B, int k, int n,
                                            int32_t* __restrict__ U, int32_t* __restrict__ count,
                                            uint32_t* __restrict__ mask, int c, int nc, uint32_t* ush) {
  __shared__ int red[kUnionNT / 64 + 1];
  const int tid = threadIdx.x;
  const int lo = c * kUnionChunk, hi = min(n, lo + kUnionChunk);
  const int n16 = (n + 15) & ~15;
  uint8_t* mk = reinterpret_cast<uint8_t*>(ush);
  uint32_t* mw = ush + n16 / 4;
  const int nq = ((hi + 15) & ~15) / 16;   // marks read below: [0, round_up(hi, 16))
  for (int q = tid; q < nq; q += kUnionNT) reinterpret_cast<uint4*>(mk)[q] = make_uint4(0u, 0u, 0u, 0u);
  if (MASK)
    for (int i = tid; i < kUnionChunk; i += kUnionNT) mw[i] = 0u;
  __syncthreads();
  union_scan(sets, B * k, [&](int e, int v) {
    if ((unsigned)v < (unsigned)hi) {
      mk[v] = 1;
      if (MASK && v >= lo) atomicOr(&mw[v - lo], 1u << (e / k));
    }
  });
  __syncthreads();
  // members before the chunk (lo is a multiple of 16)
  int part = 0;
  for (int q = tid; q < lo / 16; q += kUnionNT) {
    const uint4 w = reinterpret_cast<const uint4*>(mk)[q];
    part += byte_flags(w.x) + byte_flags(w.y) + byte_flags(w.z) + byte_flags(w.w);
  }
  int before = 0;
  (void)block_excl_scan<kUnionNT>(part, red, &before);
  // thread t ranks indices lo + 2t and lo + 2t + 1
  const int i0 = lo + 2 * tid;
  const int f0 = i0 < hi ? mk[i0] : 0, f1 = i0 + 1 < hi ? mk[i0 + 1] : 0;
  int in_chunk = 0;
  const int r = before + block_excl_scan<kUnionNT>(f0 + f1, red, &in_chunk);
  if (f0) {
    U[r] = i0;
    if (MASK) mask[r] = mw[i0 - lo];
  }
  if (f1) {
    U[r + f0] = i0 + 1;
    if (MASK) mask[r + f0] = mw[i0 + 1 - lo];
  }
  if (c == nc - 1 && tid == 0) *count = before + in_chunk;
}

template <bool MASK>
__global__ void __launch_bounds__(kUnionNT) k_union(const int32_t* __restrict__ sets, int B, int k, int n,
                                                    int32_t* __restrict__ U, int32_t* __restrict__ count,
                                                    uint32_t* __restrict__ mask) {
  extern __shared__ __attribute__((aligned(16))) uint32_t ush[];
  union_chunk<MASK>(sets, B, k, n, U, count, mask, blockIdx.x, gridDim.x, ush);
}

size_t union_lds_bytes(int n) { return (size_t)((n + 15) & ~15) + (size_t)kUnionChunk * 4; }

hipError_t launch_union(const int32_t* sets, int B, int k, int n, int32_t* U, int32_t* count, uint32_t* mask,
                        hipStream_t st) {
  const int nc = (n + kUnionChunk - 1) / kUnionChunk;
  const size_t lds = union_lds_bytes(n);
  const void* kern = mask != nullptr ? reinterpret_cast<const void*>(k_union<true>)
                                     : reinterpret_cast<const void*>(k_union<false>);
  const hipError_t e = ensure_dyn_lds(kern, lds);
  if (e != hipSuccess) return e;
  if (mask != nullptr)
    launch_k(k_union<true>, dim3(nc), dim3(kUnionNT), lds, st, sets, B, k, n, U, count, mask);
  else
    launch_k(k_union<false>, dim3(nc), dim3(kUnionNT), lds, st, sets, B, k, n, U, count, mask);
  return hipGetLastError();
}

// --------------------------------------------------------------- x-hat cast
// X16[b][0..Kpad) = fp16(LN(x[b])) (g == NULL: x[b]) for b < B; zero for b >= B
// and for k >= d. One workgroup per row b of NB; d % 4 == 0, so rows move as float4.
__device__ __forceinline__ void ln_cast_row(const float* __restrict__ x, int B, int d, int Kpad,
                                            const float* __restrict__ g, const float* __restrict__ be, float eps,
                                            _Float16* __restrict__ X16, int b) {
  __shared__ float red[16];
  _Float16* o = X16 + (size_t)b * Kpad;
  const int n4 = d >> 2;
  if (b >= B) {
    for (int k = threadIdx.x; k < Kpad; k += 1024) o[k] = (_Float16)0.f;
    return;
  }
  const f32x4* xr = reinterpret_cast<const f32x4*>(x + (size_t)b * d);
  float mean = 0.f, rstd = 1.f;
  if (g != nullptr) {
    float sum = 0.f;
    for (int i = threadIdx.x; i < n4; i += 1024) {
      const f32x4 v = xr[i];
      sum += (v[0] + v[1]) + (v[2] + v[3]);
    }
    mean = block_sum<1024>(sum, red) / (float)d;
    float q = 0.f;
    for (int i = threadIdx.x; i < n4; i += 1024) {
      const f32x4 v = xr[i];
      const float a0 = v[0] - mean, a1 = v[1] - mean, a2 = v[2] - mean, a3 = v[3] - mean;
      q += (a0 * a0 + a1 * a1) + (a2 * a2 + a3 * a3);
    }
    rstd = 1.0f / sqrtf(block_sum<1024>(q, red) / (float)d + eps);
  }
  for (int i = threadIdx.x; i < (Kpad >> 2); i += 1024) {
    f32x4 v = {0.f, 0.f, 0.f, 0.f};
    if (i < n4) {
      v = xr[i];
      if (g != nullptr) {
        const f32x4 gg = reinterpret_cast<const f32x4*>(g)[i];
        const f32x4 bb = be ? reinterpret_cast<const f32x4*>(be)[i] : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = (v[e] - mean) * rstd * gg[e] + bb[e];
      }
    }
    typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
    f16x4 h;
#pragma unroll
    for (int e = 0; e < 4; ++e) h[e] = (_Float16)v[e];
    reinterpret_cast<f16x4*>(o)[i] = h;
  }
}

__global__ void __launch_bounds__(1024) k_ln_cast(const float* __restrict__ x, int B, int d, int Kpad,
                                                  const float* __restrict__ g, const float* __restrict__ be,
                                                  float eps, _Float16* __restrict__ X16) {
  ln_cast_row(x, B, d, Kpad, g, be, eps, X16, blockIdx.x);
}

// The cast and the union of the batch's sets in one launch (they are independent):
// workgroups [0, NB) cast row b, the next nc take union chunk c.
template <bool MASK>
__global__ void __launch_bounds__(1024) k_cast_union(const float* __restrict__ x, int B, int d, int Kpad,
                                                     const float* __restrict__ g, const float* __restrict__ be,
                                                     float eps, _Float16* __restrict__ X16, int NB,
                                                     const int32_t* __restrict__ sets, int k, int n,
                                                     int32_t* __restrict__ U, int32_t* __restrict__ count,
                                                     uint32_t* __restrict__ mask, int nc) {
  extern __shared__ __attribute__((aligned(16))) uint32_t ush[];
  if ((int)blockIdx.x < NB)
    ln_cast_row(x, B, d, Kpad, g, be, eps, X16, blockIdx.x);
  else
    union_chunk<MASK>(sets, B, k, n, U, count, mask, (int)blockIdx.x - NB, nc, ush);
}

hipError_t launch_ln_cast(const float* x, int B, int NB, int d, int Kpad, const float* g, const float* be, float eps,
                          _Float16* X16, hipStream_t st) {
  launch_k(k_ln_cast, dim3(NB), dim3(1024), 0, st, x, B, d, Kpad, g, be, eps, X16);
  return hipGetLastError();
}

hipError_t launch_cast_union(const float* x, int B, int NB, int d, int Kpad, const float* g, const float* be,
                             float eps, _Float16* X16, const int32_t* sets, int k, int n, int32_t* U,
                             int32_t* count, uint32_t* mask, hipStream_t st) {
  static_assert(kUnionNT == 1024, "the cast and the union share the workgroup size");
  const int nc = (n + kUnionChunk - 1) / kUnionChunk;
  const size_t lds = union_lds_bytes(n);
  const void* kern = mask != nullptr ? reinterpret_cast<const void*>(k_cast_union<true>)
                                     : reinterpret_cast<const void*>(k_cast_union<false>);
  const hipError_t e = ensure_dyn_lds(kern, lds);
  if (e != hipSuccess) return e;
  if (mask != nullptr)
    launch_k(k_cast_union<true>, dim3(NB + nc), dim3(1024), lds, st, x, B, d, Kpad, g, be, eps, X16, NB,
                       sets, k, n, U, count, mask, nc);
  else
    launch_k(k_cast_union<false>, dim3(NB + nc), dim3(1024), lds, st, x, B, d, Kpad, g, be, eps, X16, NB,
                       sets, k, n, U, count, mask, nc);
  return hipGetLastError();
}

// ------------------------------------------------------------ k_mfma_rows
template <int MODE>
__device__ __forceinline__ int rows_count(const MrowsArgs& a) {
  if constexpr (MODE == kRowsIdentity) {
    return a.nrows;
  } else {
    const int c = a.list_count ? min(*a.list_count, a.list_max) : a.list_max;
    return MODE == kRowsList ? c : 3 * c * a.dh;
  }
}

// Rows are addressed in two steps so that the index load of a tile can be issued well
// ahead: rows_key(r) loads the list entry row r depends on (nothing for identity
// rows), rows_addr(r, key) forms the address without further loads.
template <int MODE>
__device__ __forceinline__ int rows_key(const MrowsArgs& a, int r, int nrows) {
  if constexpr (MODE == kRowsIdentity) {
    return 0;
  } else if constexpr (MODE == kRowsList) {
    return a.list[r];
  } else {
    const int per = nrows / 3;
    return a.list[(r % per) / a.dh];
  }
}
template <int MODE>
__device__ __forceinline__ const char* rows_addr(const MrowsArgs& a, int r, int key, int nrows) {
  if constexpr (MODE == kRowsIdentity) {
    return r < a.n0 ? static_cast<const char*>(a.W0) + (size_t)r * a.d * 2
                    : static_cast<const char*>(a.W1) + (size_t)(r - a.n0) * a.d * 2;
  } else {
    const int k = min(max(key, 0), a.list_range - 1);
    if constexpr (MODE == kRowsList) {
      return static_cast<const char*>(a.W0) + (size_t)k * a.d * 2;
    } else {
      const int per = nrows / 3;
      const int m = r / per;
      const int t = (r - m * per) % a.dh;
      const void* W = m == 0 ? a.W0 : (m == 1 ? a.W1 : a.W2);
      return static_cast<const char*>(W) + ((size_t)k * a.dh + t) * a.d * 2;
    }
  }
}

constexpr int kMrTiles = 10;   // tiles a wavefront accumulates in registers at a time

// One workgroup per CU. Per wavefront and 16-row tile, each load instruction fetches
// whole 128-byte lines (8 rows x 8 lanes x 16 bytes): fetching the MFMA operand layout
// straight from memory (16 rows x 64 bytes per instruction) runs at about 70% of the
// bandwidth of whole-line loads. Each 64-element block of the tile's 16 rows is then
// re-laid through a 2 KB per-wavefront LDS tile (16-byte chunk c of row r stored at
// c ^ (r & 7), conflict-free both ways) into the A operand: lane (lr, lg) takes row lr,
// chunk 4h + lg for k-step h of the block, which is exactly the k-range the B operand
// (x-hat from LDS) supplies for that lane group.
template <int NB, int NW, int U, int MODE>
__global__ void __launch_bounds__(NW * 64) k_mfma_rows(MrowsArgs a) {
  static_assert(U % 2 == 0, "a batch is whole 64-element blocks");
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

  const int n = rows_count<MODE>(a);
  const int ntiles = (n + 15) >> 4;
  const int wave = tid >> 6, lane = tid & 63;
  const int lr = lane & 15, lg = lane >> 4;
  _Float16* at = xs + NB * ldx + wave * (16 * 64);    // this wavefront's re-layout tile
  const int tstride = G * NW;
  int tile = g * NW + wave;
  if (tile >= ntiles) return;                    // no barrier follows
  const int nbat = a.Ks / (32 * U);              // batches of U instructions (U/2 blocks)
  const int kvalid = min(a.Ks, a.d - k0) * 2;    // valid bytes of this split in a row (>= 16)
  const int cb = (lane & 7) * 16;                // this lane's 16 bytes of a 128-byte block
  const int rl0 = lane >> 3, rl1 = 8 + (lane >> 3);   // its rows of a tile (even / odd loads)

  auto key_of = [&](int t, int rl) { return rows_key<MODE>(a, min(t * 16 + rl, n - 1), n); };
  // One batch: U loads of tile t's rows (chunks past the row or past n are clamped,
  // in-bounds loads, zeroed only when written to LDS, so that no select waits on a
  // load right after issuing it), then its U/2 blocks re-laid and multiplied.
  auto batch = [&](int t, int key0, int key1, int bi, f32x4 (&acc)[NBT]) {
    const int r0 = t * 16 + rl0, r1 = t * 16 + rl1;
    const char* p0 = rows_addr<MODE>(a, min(r0, n - 1), key0, n) + k0 * 2;
    const char* p1 = rows_addr<MODE>(a, min(r1, n - 1), key1, n) + k0 * 2;
    u32x4 w[U];
    unsigned okm = 0u;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int off = (bi * (U / 2) + (u >> 1)) * 128 + cb;
      okm |= (off < kvalid && ((u & 1) ? r1 : r0) < n) ? (1u << u) : 0u;
      w[u] = ld_stream(((u & 1) ? p1 : p0) + min(off, kvalid - 16));
    }
#pragma unroll
    for (int blk = 0; blk < U / 2; ++blk) {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int r = rl0 + 8 * i, c = lane & 7;
        const int u = 2 * blk + i;
        *reinterpret_cast<u32x4*>(at + r * 64 + ((c ^ (r & 7)) << 3)) =
            ((okm >> u) & 1u) ? w[u] : u32x4{0u, 0u, 0u, 0u};
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int c = 4 * h + lg;
        const f16x8 av = *reinterpret_cast<const f16x8*>(at + lr * 64 + ((c ^ (lr & 7)) << 3));
        const int ks = 2 * (bi * (U / 2) + blk) + h;
#pragma unroll
        for (int j = 0; j < NBT; ++j) {
          const f16x8 bv = *reinterpret_cast<const f16x8*>(xs + (lr + 16 * j) * ldx + 32 * ks + 8 * lg);
          acc[j] = mfma16x16x32(av, bv, acc[j]);
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
  };
  // This wavefront's tiles are tile, tile + tstride, ...; up to kMrTiles of them at a time
  // keep their accumulators in registers, and their results are written once all of
  // them are done. Written per tile instead, the partials (a few hundred bytes per
  // wavefront, every few microseconds) interleave DRAM writes with the weight stream,
  // which cost far more than their bytes: at batch 32, QKV 175 us against 142 us with
  // the stores kept in L2. Each tile's rows are read to the end of the split before the
  // next tile starts (QKV at batch 32: 154 us, against 161-167 us with the batch loop
  // outside, which jumps between tiles every 512 bytes of a row).
  const int mine = (ntiles - tile + tstride - 1) / tstride;
  for (int c0 = 0; c0 < mine; c0 += kMrTiles) {
    int key0[kMrTiles], key1[kMrTiles];
#pragma unroll
    for (int q = 0; q < kMrTiles; ++q) {
      const int t = tile + min(c0 + q, mine - 1) * tstride;   // (clamped, unconditional)
      key0[q] = key_of(t, rl0);
      key1[q] = key_of(t, rl1);
    }
    f32x4 acc[kMrTiles][NBT];
#pragma unroll
    for (int q = 0; q < kMrTiles; ++q)
#pragma unroll
      for (int j = 0; j < NBT; ++j) acc[q][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < kMrTiles; ++q)
      if (c0 + q < mine)
        for (int bi = 0; bi < nbat; ++bi) batch(tile + (c0 + q) * tstride, key0[q], key1[q], bi, acc[q]);
#pragma unroll
    for (int q = 0; q < kMrTiles; ++q) {
      if (c0 + q >= mine) continue;
      const int t = tile + (c0 + q) * tstride;
      // lane holds rows t*16 + 4*lg + i, token columns lr + 16*j
      if (a.out0 != nullptr) {
#pragma unroll
        for (int j = 0; j < NBT; ++j) {
          const int b = lr + 16 * j;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int r = t * 16 + 4 * lg + i;
            if (r < n && b < a.B) {
              if (r < a.n0) a.out0[(size_t)b * a.ld0 + r] = acc[q][j][i];
              else a.out1[(size_t)b * a.ld1 + (r - a.n0)] = acc[q][j][i];
            }
          }
        }
      } else {
        // whole rows of NB floats with 16-byte stores, through the wavefront's LDS tile
        float* tf = reinterpret_cast<float*>(at);        // [16][NB] fp32 (<= the 2 KB tile)
#pragma unroll
        for (int j = 0; j < NBT; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i) tf[(4 * lg + i) * NB + lr + 16 * j] = acc[q][j][i];
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        constexpr int LPRW = NB / 4, RPI = 64 / LPRW;   // lanes per row, rows per instruction
        const int cq = 4 * (lane % LPRW);
#pragma unroll
        for (int rr = lane / LPRW; rr < 16; rr += RPI) {
          const int r = t * 16 + rr;
          if (r < n)
            *reinterpret_cast<f32x4*>(a.P + ((size_t)s * a.nrows_pad + r) * NB + cq) =
                *reinterpret_cast<const f32x4*>(tf + rr * NB + cq);
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      }
    }
  }
}

// K per split for k_mfma_rows: a multiple of 32 * kMrU halves whose staged slice of
// NB rows fits 96 KB of LDS (with the re-layout tiles, one workgroup per CU).
static constexpr int kMrU = 8, kMrNW = 8;
static constexpr int kMrTileBytes = kMrNW * 16 * 64 * 2;
void mrows_split(int Kpad, int NB, int* S, int* Ks) {
  const int budget = min(device_lds_per_block() - kMrTileBytes, 98304 + NB * 16);
  const int unit = 32 * kMrU;
  int kmax = ((budget / (NB * 2) - 8) / unit) * unit;
  if (kmax < unit) kmax = unit;
  int s = (Kpad + kmax - 1) / kmax;
  int ks = (((Kpad + s - 1) / s) + unit - 1) / unit * unit;
  *S = s;
  *Ks = ks;
}

template <int NB, int MODE>
static hipError_t launch_mrows_t(MrowsArgs a, hipStream_t st) {
  const size_t lds = (size_t)NB * (a.Ks + 8) * 2 + kMrTileBytes;
  const auto kern = k_mfma_rows<NB, kMrNW, kMrU, MODE>;
  const hipError_t e = ensure_dyn_lds(reinterpret_cast<const void*>(kern), lds);
  if (e != hipSuccess) return e;
  const int G = max(1, device_cu_count() / a.S);
  launch_k(kern, dim3(G * a.S), dim3(kMrNW * 64), lds, st, a);
  return hipGetLastError();
}

template <int NB>
static hipError_t launch_mrows_nb(const MrowsArgs& a, hipStream_t st) {
  switch (a.mode) {
    case kRowsList: return launch_mrows_t<NB, kRowsList>(a, st);
    case kRowsHeads: return launch_mrows_t<NB, kRowsHeads>(a, st);
    default: return launch_mrows_t<NB, kRowsIdentity>(a, st);
  }
}

hipError_t launch_mrows(int NB, const MrowsArgs& a, hipStream_t st) {
  return NB <= 16 ? launch_mrows_nb<16>(a, st) : launch_mrows_nb<32>(a, st);
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
// chunk c ^ (2 * ((r >> 3) & 3)) so that the row-wise 16-byte writes are free of bank
// conflicts and the four 8-row groups of a transpose read land in distinct banks.
//
// Load pipeline of a wavefront: the row indices of batch k+2, the weights and
// coefficients of batch k+1 and the MFMAs of batch k are in flight together. Indices
// are always loaded one batch before the weights that need them, so no wait for an
// index ever drains the weight loads behind it.
template <int NB, int U>
struct ColsStep {
  u32x4 w[U][4];        // weights: rows (lane >> 3) + 8*i, 16-byte chunk lane & 7
  u32x4 h[U][NB / 16];  // coefficients: token lr + 16*j, rows 8*lg .. 8*lg + 7
  unsigned ok;          // bit 4u + i: weight chunk w[u][i] is wanted (else written as 0)
};

// Row of M for contraction row `row` (clamped into [0, uend) so that every load is in
// bounds; rows past uend are zeroed after the load).
template <bool HEADS, int U>
__device__ __forceinline__ void mc_index(int (&ix)[U][4], const McolsArgs& a, int q0, int qstride, int uend,
                                         int lane) {
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = min(32 * (q0 + u * qstride) + (lane >> 3) + 8 * i, uend - 1);
      if (HEADS) {
        const int p = row / a.dh;
        ix[u][i] = min(max(a.list[p], 0), a.list_range - 1) * a.dh + (row - p * a.dh);
      } else {
        ix[u][i] = min(max(a.list[row], 0), a.list_range - 1);
      }
    }
}

template <int NB, int U>
__device__ __forceinline__ void mc_load(ColsStep<NB, U>& st, const int (&ix)[U][4], const McolsArgs& a,
                                        const char* Mb, int q0, int qstride, int uend, bool col_on, int lane) {
  const int lr = lane & 15, lg = lane >> 4;
  const size_t rowb = (size_t)a.d * 2;
  st.ok = 0u;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int q = min(q0 + u * qstride, (uend - 1) >> 5);     // clamped: loads stay in bounds
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 32 * (q0 + u * qstride) + (lane >> 3) + 8 * i;
      st.ok |= (col_on && row < uend) ? (1u << (4 * u + i)) : 0u;
      st.w[u][i] = ld_stream(Mb + (size_t)ix[u][i] * rowb);
    }
#pragma unroll
    for (int j = 0; j < NB / 16; ++j) st.h[u][j] = ld_plain(a.C + coef_index(lr + 16 * j, 32 * q + 8 * lg, NB));
  }
}

// WIDE: the wavefronts of a workgroup take adjacent 64-column tiles over the same rows
// (each row is then read in NW * 128 contiguous bytes, and the coefficients are shared
// through L1), and each writes its own partial tile. Otherwise they split the rows of
// one 64-column tile and are summed in LDS.
template <int NB, int NW, int U, bool HEADS, bool WIDE>
__global__ void __launch_bounds__(NW * 64) k_mfma_cols(McolsArgs a) {
  constexpr int NBT = NB / 16;
  extern __shared__ __attribute__((aligned(16))) _Float16 csm[];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int lr = lane & 15, lg = lane >> 4;
  _Float16* tile = csm + wave * (32 * 64);
  float* red = reinterpret_cast<float*>(csm + NW * 32 * 64);     // [NW][NB][64] (not WIDE)
  const int n0 = WIDE ? (blockIdx.x * NW + wave) * 64 : blockIdx.x * 64;
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

  const int qstride = WIDE ? 1 : NW;
  const int bstep = qstride * U;                 // k-steps per batch of this wavefront
  int q = WIDE ? qbeg : qbeg + wave;
  if (q < qend) {
    int ix0[U][4], ix1[U][4];
    mc_index<HEADS, U>(ix0, a, q, qstride, uend, lane);
    mc_index<HEADS, U>(ix1, a, q + bstep, qstride, uend, lane);
    ColsStep<NB, U> cur;
    mc_load<NB, U>(cur, ix0, a, Mb, q, qstride, uend, col_on, lane);
  for (; q < qend; q += bstep) {
    ColsStep<NB, U> nxt;
    const bool more = q + bstep < qend;
    // issued unconditionally (clamped in-bounds past the end, then discarded) so that
    // the waits below never have to drain them
    mc_index<HEADS, U>(ix0, a, q + 2 * bstep, qstride, uend, lane);          // batch k+2
    mc_load<NB, U>(nxt, ix1, a, Mb, q + bstep, qstride, uend, col_on, lane);  // batch k+1
    __builtin_amdgcn_sched_barrier(0);          // keep the prefetch ahead of the MFMAs
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (q + u * qstride >= qend) break;
      // row-wise write of the 32 x 64 tile
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = (lane >> 3) + 8 * i;
        const int c = (lane & 7) ^ (2 * i);
        *reinterpret_cast<u32x4*>(tile + r * 64 + c * 8) =
            ((cur.ok >> (4 * u + i)) & 1u) ? cur.w[u][i] : u32x4{0u, 0u, 0u, 0u};
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      f16x8 hv[NBT];
#pragma unroll
      for (int j = 0; j < NBT; ++j) hv[j] = __builtin_bit_cast(f16x8, cur.h[u][j]);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        // Column-wise B operand (lane (n = lr, g = lg) takes rows 8g .. 8g + 7 of column
        // 16t + n) with two LDS transpose reads. Within a 16-lane group the transpose
        // read hands lane i, slot j element i % 4 of the 4 elements that lane 4j + i/4
        // addressed, so lane s addresses row 8g + s/4 (+ 4 for the second read) at
        // columns 16t + 4 (s % 4) .. + 3.
        const int col = 16 * t + 4 * (lr & 3);
        v4s_t half[2];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const int r = 8 * lg + (lr >> 2) + 4 * hh;
          const int pc = (col >> 3) ^ (2 * ((r >> 3) & 3));
          half[hh] = ds_read_tr16(tile + r * 64 + pc * 8 + (col & 7));
        }
        const f16x8 bv = __builtin_shufflevector(__builtin_bit_cast(f16x4_t, half[0]),
                                                 __builtin_bit_cast(f16x4_t, half[1]), 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
        for (int j = 0; j < NBT; ++j) acc[j][t] = mfma16x16x32(hv[j], bv, acc[j][t]);
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    if (!more) break;
    cur = nxt;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int i = 0; i < 4; ++i) ix1[u][i] = ix0[u][i];
  }
  }
  if constexpr (WIDE) {
    // lane holds tokens 16j + 4lg + i of columns n0 + 16t + lr
#pragma unroll
    for (int j = 0; j < NBT; ++j)
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int b = 16 * j + 4 * lg + i, c = n0 + 16 * t + lr;
          if (b < a.B && c < a.d) a.P[((size_t)s * a.B + b) * a.d + c] = acc[j][t][i];
        }
    return;
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

static constexpr int kMcNW = 8, kMcU = 1;
static constexpr bool kMcWide = true;

int mcols_split(int d, int nmax) {
  // one workgroup per CU: more splits only add partial-sum traffic (each split writes a
  // full B x d partial) and, past the CU count, a second round of workgroups (measured at
  // d = 12288: 10 splits 57 + 5 us out-proj, 32 splits 71 + 9 us)
  const int tiles = kMcWide ? (d + 64 * kMcNW - 1) / (64 * kMcNW) : (d + 63) / 64;
  int s = max(1, device_cu_count() / tiles);
  const int q = (nmax + 31) / 32;                  // k-steps available
  s = max(1, min(s, max(1, kMcWide ? q / 2 : q / (2 * kMcNW))));
  return min(s, 32);
}

template <int NB>
static hipError_t launch_mcols_t(const McolsArgs& a, hipStream_t st) {
  const size_t lds = (size_t)kMcNW * 32 * 64 * 2 + (kMcWide ? 0 : (size_t)kMcNW * NB * 64 * 4);
  dim3 grid(kMcWide ? (a.d + 64 * kMcNW - 1) / (64 * kMcNW) : (a.d + 63) / 64, a.S);
  if (a.dh > 0)
    launch_k((k_mfma_cols<NB, kMcNW, kMcU, true, kMcWide>), grid, dim3(kMcNW * 64), lds, st, a);
  else
    launch_k((k_mfma_cols<NB, kMcNW, kMcU, false, kMcWide>), grid, dim3(kMcNW * 64), lds, st, a);
  return hipGetLastError();
}

hipError_t launch_mcols(int NB, const McolsArgs& a, hipStream_t st) {
  return NB <= 16 ? launch_mcols_t<16>(a, st) : launch_mcols_t<32>(a, st);
}

// --------------------------------------------------------------- finishers
// sum_{s < S} P[s * stride + e] in split order, with up to 8 loads in flight.
// Four consecutive elements summed over the splits in split order (the same order, so
// the same bits, as sum_splits per element); every split's load is issued before the
// first add, unpredicated (split index clamped, surplus not added).
__device__ __forceinline__ f32x4 sum_splits4(const float* __restrict__ P, int S, size_t stride, size_t e) {
  f32x4 v = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < S; s0 += 8) {
    f32x4 t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) t[u] = *reinterpret_cast<const f32x4*>(P + (size_t)min(s0 + u, S - 1) * stride + e);
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (s0 + u < S) v += t[u];
  }
  return v;
}

__device__ __forceinline__ float sum_splits(const float* __restrict__ P, int S, size_t stride, size_t e) {
  float v = 0.f;
  for (int s0 = 0; s0 < S; s0 += 8) {
    float t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) t[u] = s0 + u < S ? P[(size_t)(s0 + u) * stride + e] : 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) v += t[u];
  }
  return v;
}

// fc1: C(b, u) = fp16(ReLU(sum_s P[s][u][b] + b1[list[u]])) for b < B and u < n (and,
// with a mask, only where bit b of mask[u] is set); zero elsewhere up to a multiple
// of 64 rows. One workgroup per 64 rows.
template <int NB>
__global__ void __launch_bounds__(16 * NB) k_fc1_finish(Fc1FinishArgs a) {
  // one thread per four tokens of one of the workgroup's 64 rows: a single round trip
  __shared__ float t[64][NB + 1];
  const int n = a.list_count ? min(*a.list_count, a.list_max) : a.list_max;
  const int u0 = blockIdx.x * 64;
  if (u0 >= ((n + 63) & ~63)) return;
  {
    const int ul = threadIdx.x / (NB / 4), b0 = (threadIdx.x - ul * (NB / 4)) * 4;
    const int u = u0 + ul;
    f32x4 v = {0.f, 0.f, 0.f, 0.f};
    if (u < n) {
      v = sum_splits4(a.P, a.S, (size_t)a.nrows_pad * NB, (size_t)u * NB + b0);
      const float bias = a.b1 ? a.b1[min(max(a.list[u], 0), a.list_range - 1)] : 0.f;
      const uint32_t mk = a.mask ? a.mask[u] : 0xffffffffu;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float x = v[i] + bias;
        x = act_apply(x, a.act);
        if (b0 + i >= a.B || !((mk >> (b0 + i)) & 1u)) x = 0.f;
        v[i] = x;
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) t[ul][b0 + i] = v[i];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < 64 * NB; e += 16 * NB) {
    const int b = e >> 6, ul = e & 63;
    a.C[coef_index(b, u0 + ul, NB)] = (_Float16)t[ul][b];
  }
}

hipError_t launch_fc1_finish(int NB, const Fc1FinishArgs& a, hipStream_t st) {
  const int blocks = max(1, (a.list_max + 63) / 64);
  if (NB <= 16)
    launch_k(k_fc1_finish<16>, dim3(blocks), dim3(16 * 16), 0, st, a);
  else
    launch_k(k_fc1_finish<32>, dim3(blocks), dim3(16 * 32), 0, st, a);
  return hipGetLastError();
}

// Sum of k_mfma_cols partials: out[b][c] = sum_s P2[s][b][c] + bias[c] + resid[b][c];
// one thread per four columns (d % 4 == 0), every split's load in flight at once.
__global__ void __launch_bounds__(256) k_cols_finish(ColsFinishArgs a) {
  const long total = (long)a.B * a.d;
  const long e = ((long)blockIdx.x * 256 + threadIdx.x) * 4;
  if (e >= total) return;
  const int c = (int)(e % a.d);
  f32x4 v = sum_splits4(a.P, a.S, (size_t)total, (size_t)e);
  if (a.bias) v += *reinterpret_cast<const f32x4*>(a.bias + c);
  if (a.resid) v += *reinterpret_cast<const f32x4*>(a.resid + e);
  *reinterpret_cast<f32x4*>(a.out + e) = v;
}

hipError_t launch_cols_finish(const ColsFinishArgs& a, hipStream_t st) {
  const long quads = ((long)a.B * a.d / 4 + 255) / 256;
  launch_k(k_cols_finish, dim3((unsigned)max(1L, quads)), dim3(256), 0, st, a);
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
    if (b < B && j < r) v = sum_splits(P, S, (size_t)nrows_pad * NB, (size_t)(row0 + j) * NB + b);
    C[e] = (_Float16)v;
  }
}

hipError_t launch_sum_cast(int NB, const float* P, int S, int nrows_pad, int row0, int r, int B, _Float16* C, int ldc,
                           hipStream_t st) {
  const int blocks = min((NB * ldc + 255) / 256, 4 * device_cu_count());
  if (NB <= 16)
    launch_k(k_sum_cast<16>, dim3(blocks), dim3(256), 0, st, P, S, nrows_pad, row0, r, B, C, ldc);
  else
    launch_k(k_sum_cast<32>, dim3(blocks), dim3(256), 0, st, P, S, nrows_pad, row0, r, B, C, ldc);
  return hipGetLastError();
}

// Q/K/V of the batch. One workgroup per (union head p, projection m): the dh x NB
// partial sums of its rows are read contiguously, summed over the splits in order and
// biased; then for every sequence b whose set holds h = list[p] (as its j-th head) the
// query goes to q[b][j][:] (m = 0) or the key/value to cache row pos[b] of head h
// (m = 1, 2; round to nearest even).
template <int NB, typename KT>
__global__ void __launch_bounds__(1024) k_qkv_finish(QkvFinishArgs a) {
  extern __shared__ float qsm[];                  // [dh][NB + 1]
  __shared__ int jsel[NB];
  const int p = blockIdx.x, m = blockIdx.y;
  if (a.zero != nullptr) {   // the attention's coefficient matrix, before it writes its part
    const int wg = blockIdx.x + gridDim.x * blockIdx.y, nwg = gridDim.x * gridDim.y;
    for (int i = wg * 1024 + (int)threadIdx.x; i < a.zero_n / 8; i += nwg * 1024)
      reinterpret_cast<u32x4*>(a.zero)[i] = u32x4{0u, 0u, 0u, 0u};
  }
  const int nu = *a.hcount;
  if (p >= nu) return;
  const int h = min(max(a.hlist[p], 0), a.H - 1);
  if (threadIdx.x < NB) {
    int jj = -1;
    const int b = threadIdx.x;
    if (b < a.B) {
      const int32_t* hs = a.heads + (size_t)b * a.n_heads;
      int lo = 0, hi = a.n_heads - 1;
      while (lo <= hi) {
        const int mid = (lo + hi) >> 1;
        if (hs[mid] == h) { jj = mid; break; }
        if (hs[mid] < h) lo = mid + 1; else hi = mid - 1;
      }
    }
    jsel[b] = jj;
  }
  const size_t r0 = ((size_t)m * nu + p) * a.dh;
  const float* bias = m == 0 ? a.bq : (m == 1 ? a.bk : a.bv);
  // one thread per four tokens of a row: every split's load in flight at once
  for (int e = threadIdx.x * 4; e < a.dh * NB; e += 1024 * 4) {
    const int t = e / NB, b = e - t * NB;
    f32x4 v = sum_splits4(a.P, a.S, (size_t)a.nrows_pad * NB, (r0 + t) * NB + b);
    const float bs = bias ? bias[(size_t)h * a.dh + t] : 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) qsm[t * (NB + 1) + b + i] = v[i] + bs;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < a.dh * NB; e += 1024) {
    const int b = e / a.dh, t = e - b * a.dh;
    const int jj = jsel[b];
    if (jj < 0) continue;
    const float v = qsm[t * (NB + 1) + b];
    if (m == 0) {
      a.q[((size_t)b * a.n_heads + jj) * a.dh + t] = v;
    } else {
      KT* Cc = static_cast<KT*>(m == 1 ? a.K : a.V);
      Cc[(((size_t)b * a.H + h) * a.cap + a.posb[b]) * a.dh + t] = (KT)v;
    }
  }
}

hipError_t launch_qkv_finish(int NB, int kvtype, const QkvFinishArgs& a, hipStream_t st) {
  dim3 grid(a.H, 3);
  const size_t lds = (size_t)a.dh * (NB + 1) * sizeof(float);
  if (NB <= 16) {
    if (kvtype == DV_F16) launch_k((k_qkv_finish<16, _Float16>), grid, dim3(1024), lds, st, a);
    else launch_k((k_qkv_finish<16, float>), grid, dim3(1024), lds, st, a);
  } else {
    if (kvtype == DV_F16) launch_k((k_qkv_finish<32, _Float16>), grid, dim3(1024), lds, st, a);
    else launch_k((k_qkv_finish<32, float>), grid, dim3(1024), lds, st, a);
  }
  return hipGetLastError();
}

// Attention outputs as out-projection coefficients: C(b, p*dh + t) = H_h(x_b)[t] for
// the union head h = list[p] if h is in sequence b's set (combining its split-KV
// partials), else 0; rows up to ldc are covered (zero beyond the union). C is in the
// layout of coef_index with gridDim.y (the padded token count) tokens.
__global__ void __launch_bounds__(256) k_attn_finish(AttnFinishArgs a) {
  __shared__ float fac[kAttnMaxSplit];
  __shared__ int jsel;
  const int p = blockIdx.x, b = blockIdx.y;
  const int nu = *a.hcount;
  const int r0 = p * a.dh;
  if (r0 >= a.ldc) return;
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
    a.C[coef_index(b, r0 + t, gridDim.y)] = (_Float16)v;
  }
}

hipError_t launch_attn_finish(int NB, const AttnFinishArgs& a, hipStream_t st) {
  dim3 grid((a.ldc + a.dh - 1) / a.dh, NB);
  launch_k(k_attn_finish, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace dv
