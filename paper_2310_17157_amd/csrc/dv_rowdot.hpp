// Row-dot loops shared by the predictor's first layer, fc1 and the gathered QKV:
// every selected row (d weights, 16-byte chunks) is dotted with an input vector
// staged once per workgroup in LDS (optionally layer-normalised there).
#pragma once

#include "dv_internal.hpp"

namespace dv {

// Weight loads per wavefront issued before the input is staged.
constexpr int kRowdotPre = 4;

// rowdot_flat: workgroup wg of G takes the contiguous rows [wg*R/G, (wg+1)*R/G), and
// its NW wavefronts split that range's load slots evenly across row boundaries (a
// slot is one wavefront load of 64 lanes x 16 bytes; a row of nch chunks is
// ipr = ceil(nch / 64) slots). Every wavefront thus has the same number of loads
// whatever the row count: the first batch of U around the prologue (kRowdotPre
// behind the input reads, the rest once the input is staged), then each next U
// before the current U are consumed (two alternating register sets, so that no wait
// is ever needed just to move data; surplus loads past the end are clamped to the
// last slot and discarded). Callers keep U small (2): deeper queues per wavefront
// were measured slower on this part. A wavefront reduces its partial
// sum of a row when it leaves the row and records it in LDS (part[wave * mr + k] for its k-th
// row, mr = ceil(R/G) + 1); after a barrier one thread per row adds the records of the
// wavefronts that covered it, in wavefront order (bitwise reproducible), and calls
// epi(row, value). xhat_out (optional) receives the staged input from workgroup 0.
// KX: float4 of the input per thread (d <= 4 * 64 * NW * KX); LN: layer norm of the
// input with gamma g (non-NULL) and beta be (NULL: 0). tail() is called by
// every thread once its wavefront has streamed all its loads, before the barrier that
// precedes epi (a place to issue the epilogue's own reads).
struct NoTail {
  __device__ void operator()() const {}
};
// Chunk-scale rows of 4-bit weights (unused for fp16 / fp32 rows).
struct NoScales {
  __device__ const _Float16* operator()(int) const { return nullptr; }
};

// i * n / G rounded down: the boundary of part i of n rows split G ways (in 32 bits
// where the product fits, avoiding the long 64-bit division sequence).
__device__ __forceinline__ int rowdot_split(int i, int n, int G) {
  if (n < (1 << 23) && i <= 256) return (int)((unsigned)(i * n) / (unsigned)G);
  return (int)((long)i * n / G);
}
// For 4-bit rows (T = q4_t) scale_ptr(row) gives the row's chunk scales; each weight
// load is paired with the load of its chunk's scale.
template <typename T, int NW, int U, int KX, bool LN, class RowPtr, class Epi, class Tail = NoTail,
          class ScalePtr = NoScales>
__device__ __forceinline__ void rowdot_flat(RowPtr row_ptr, Epi epi, int nrows, int d, const float* x,
                                            const float* g, const float* be, float eps, float* xs, float* red,
                                            float* part, float* xhat_out, int wg, int G, Tail tail = Tail(),
                                            ScalePtr scale_ptr = ScalePtr()) {
  constexpr int NT = NW * 64;
  constexpr int E = Chunk<T>::E;
  // the input's reads go out first of all, ahead of the partition arithmetic
  StageX<T, NT, KX, LN> st;
  st.load(x, d, g, be);
  // wave-uniform: row pointers and slot bounds live in scalar registers, so that a
  // row change costs a scalar load (its own counter), never a wait on the stream
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int r0 = rowdot_split(wg, nrows, G), r1 = rowdot_split(wg + 1, nrows, G);
  const int nch = d / E, ipr = (nch + 63) >> 6;
  const int slots = (r1 - r0) * ipr;
  const int tw = (slots + NW - 1) / NW;
  const int s0 = min(wave * tw, slots), s1 = min(s0 + tw, slots);
  const int mr = (nrows + G - 1) / G + 1;
  const bool active = s0 < s1;
  // Every wavefront issues the same loads on every path (a wait after a branch that
  // skips loads is counted for the path without them, so it would also wait for the
  // loads in flight): a wavefront without slots re-reads its workgroup's last slot,
  // and in a workgroup without rows the input vector (d floats, at least one row of
  // T) stands in for a row.
  const bool any = slots > 0;
  const int shi = active ? s1 - 1 : slots - 1;   // last slot this wavefront reads

  // The row pointer (a list lookup for gathered rows) is formed only when the load
  // stream enters a new row, not per load.
  int lrow = -1;
  const char* lptr = nullptr;
  const _Float16* sptr = nullptr;   // 4-bit rows: the row's chunk scales
  constexpr bool Q4 = kIsQ4<T>;
  struct Batch {
    u32x4 w[U];
    _Float16 s[Q4 ? U : 1];
  };
  auto set_row = [&](int rr) {
    lrow = rr;
    lptr = any ? reinterpret_cast<const char*>(row_ptr(r0 + rr)) : reinterpret_cast<const char*>(x);
    if constexpr (Q4) sptr = any ? scale_ptr(r0 + rr) : reinterpret_cast<const _Float16*>(x);
  };
  // loads u in [u0, u1) of the batch of U slots starting at sb (u0, u1 compile-time)
  auto load_part = [&](Batch& b, int sb, int u0, int u1) {
    const int sc0 = max(min(sb + u0, shi), 0);
    int rr = sc0 / ipr, j = sc0 - rr * ipr;
    if (rr != lrow) set_row(rr);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (u < u0 || u >= u1) continue;
      if (u > u0 && sb + u <= shi) {
        if (++j == ipr) {
          j = 0;
          ++rr;
          set_row(rr);
        }
      }
      const int c = min(j * 64 + lane, nch - 1);
      b.w[u] = ld_stream(lptr + (size_t)c * 16);
      if constexpr (Q4) b.s[u] = sptr[c];
    }
  };
  auto load = [&](Batch& b, int sb) { load_part(b, sb, 0, U); };
  int cur = active ? s0 / ipr : 0;        // relative row being accumulated
  const int first = cur;
  float acc0 = 0.f, acc1 = 0.f;
  auto flush = [&]() {
    const float v = wave_sum(acc0 + acc1);
    if (lane == 0) part[wave * mr + (cur - first)] = v;
    acc0 = 0.f;
    acc1 = 0.f;
  };
  auto consume = [&](const Batch& b, int sb) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = sb + u;
      if (s >= s1) break;
      const int rr = s / ipr;
      if (rr != cur) {
        flush();
        cur = rr;
      }
      const int c = (s - rr * ipr) * 64 + lane;
      if (c < nch) {
        float& acc = (u & 1) ? acc1 : acc0;
        if constexpr (Q4)
          acc = dot_chunk_q4(b.w[u], (float)b.s[u], xs, d, c, acc);
        else
          acc = dot_chunk<T>(b.w[u], xs, d, c, acc);
      }
    }
  };

  // Input reads first and only PRE weight reads behind them; the rest of the first
  // batch follows once the input is staged, so that the staging reads do not queue
  // behind a full batch from every wavefront of the grid.
  constexpr int PRE = kRowdotPre < U ? kRowdotPre : U;
  Batch wa;
  if (PRE > 0) load_part(wa, s0, 0, PRE);
  st.finish(d, be != nullptr, eps, xs, red);
  if (PRE < U) load_part(wa, s0, PRE, U);
  if (xhat_out != nullptr && wg == 0)
    for (int e = threadIdx.x; e < d; e += NT) xhat_out[e] = xs[xs_index<T>(e, d)];
  if (active) {
    Batch wb;
    for (int sb = s0;;) {
      load(wb, sb + U);
      consume(wa, sb);
      sb += U;
      if (sb >= s1) break;
      load(wa, sb + U);
      consume(wb, sb);
      sb += U;
      if (sb >= s1) break;
    }
    flush();
  }
  tail();
  __syncthreads();
  for (int rr = threadIdx.x; rr < r1 - r0; rr += NT) {
    const int wa0 = (rr * ipr) / tw, wb0 = min(((rr + 1) * ipr - 1) / tw, NW - 1);
    float v = 0.f;
    for (int w = wa0; w <= wb0; ++w) v += part[w * mr + (rr - (w * tw) / ipr)];
    epi(r0 + rr, v);
  }
}

// Smallest KX for a row of d floats with NW wavefronts (at most 4).
inline int rowdot_kx(int d, int nw) { return (d + 256 * nw - 1) / (256 * nw); }

// LDS floats rowdot_flat needs for its per-wavefront records.
inline int rowdot_flat_part(int nrows, int G, int nw) { return nw * ((nrows + G - 1) / G + 1); }

}  // namespace dv
