// Workgroup-level set selection over one row of predictor scores.
//
// Top-k: the k largest scores, ties broken toward the lower index; threshold:
// every score >= t (the labelling rule of Algorithm 1). Output is ascending.
//
// Method: scores are mapped to order-preserving 32-bit keys. An MSB-first radix
// select finds the key digit by digit (13, 13, then 6 bits) with LDS histograms of
// the candidates that still match the prefix found so far; it stops as soon as the
// digit's bin holds exactly the number of elements still needed. An ordered
// compaction (two workgroup-wide exclusive scans over contiguous per-thread ranges)
// then writes the selected indices in ascending order, taking equal keys at the
// boundary lowest index first. Everything is integer work on keys, so the result is
// exact and deterministic. Score loads are coalesced and several are kept in flight,
// since the scores come from L2 and every pass is latency-bound.
#pragma once

#include <limits.h>

#include "dv_internal.hpp"

namespace dv {

constexpr int kSelBins = 8192;   // LDS histogram bins (13-bit digits)

// Scratch ints needed by the selection routines for an NT-thread workgroup.
constexpr int kSelSm(int NT) { return 2 * (NT / 64) + 8; }

__device__ __forceinline__ uint32_t shr32(uint32_t v, int s) { return s >= 32 ? 0u : (v >> s); }

// Find the digit holding the krem-th largest candidate: bins above it hold `above`
// (< krem) candidates, and above + hist[digit] >= krem. sm: >= NT/64 + 2 ints.
template <int NT>
__device__ __forceinline__ void find_digit(const uint32_t* hist, int nb, int krem, int* sm,
                                           int* digit, int* above) {
  const int R = (nb + NT - 1) / NT;
  const int b0 = threadIdx.x * R;
  int local = 0;
  for (int j = 0; j < R; ++j)
    if (b0 + j < nb) local += (int)hist[b0 + j];
  int tot;
  const int pre = block_excl_scan<NT>(local, sm, &tot);
  const int suffix = tot - pre - local;   // candidates in bins owned by higher threads
  if (suffix < krem && krem <= suffix + local) {
    int run = suffix;
    for (int j = R - 1; j >= 0; --j) {
      const int b = b0 + j;
      if (b >= nb) continue;
      const int c = (int)hist[b];
      if (run + c >= krem) {
        sm[NT / kWave] = b;
        sm[NT / kWave + 1] = run;
        break;
      }
      run += c;
    }
  }
  __syncthreads();
  *digit = sm[NT / kWave];
  *above = sm[NT / kWave + 1];
}

// Select over s[0..n). Writes the set to out[0..min(count, cap)) (and out2 if not
// NULL) and the set size to *count_out (if not NULL). hist: kSelBins u32 of LDS;
// sm: kSelSm(NT) ints of LDS. Called by the whole workgroup.
template <int NT>
__device__ void wg_select(const float* __restrict__ s, int n, int mode, int k, float thresh,
                          int32_t* __restrict__ out, int cap, int32_t* __restrict__ count_out,
                          int32_t* __restrict__ out2, uint32_t* hist, int* sm) {
  const int tid = threadIdx.x;
  uint32_t prefix = 0u;
  int pbits = 0;
  int eq_take = INT_MAX;
  bool all = false;
  if (mode == DV_SELECT_THRESHOLD) {
    prefix = fkey(thresh);
    pbits = 32;
  } else if (k >= n) {
    all = true;
  } else if (k <= 0) {
    if (tid == 0 && count_out) *count_out = 0;
    return;
  } else {
    int krem = k;
    for (int p = 0; p < 3; ++p) {
      const int D = p < 2 ? 13 : 6, nb = 1 << D;   // 13 + 13 + 6 = 32 key bits
      for (int i = tid; i < nb; i += NT) hist[i] = 0u;
      __syncthreads();
      const int lo = 32 - pbits - D;
      const int hi = 32 - pbits;
      for (int b = 0; b < n; b += NT * 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int i = b + u * NT + tid;
          v[u] = i < n ? s[i] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const uint32_t key = fkey(v[u]);
          if (b + u * NT + tid < n && (pbits == 0 || shr32(key, hi) == prefix))
            atomicAdd(&hist[(key >> lo) & (uint32_t)(nb - 1)], 1u);
        }
      }
      __syncthreads();
      int dig, above;
      find_digit<NT>(hist, nb, krem, sm, &dig, &above);
      const int cnt = (int)hist[dig];
      krem -= above;
      prefix = (prefix << D) | (uint32_t)dig;
      pbits += D;
      __syncthreads();
      if (cnt == krem) {          // the whole bin is selected: a strict key prefix test suffices
        eq_take = INT_MAX;
        break;
      }
      eq_take = krem;             // ties at the full key: lowest indices first
    }
  }

  // Ordered compaction. Wavefront w owns the contiguous segment [w*seg, (w+1)*seg)
  // and walks it 64 scores at a time (coalesced loads, kUnroll in flight); ranks
  // within a group come from ballots, across groups from running counts, across
  // wavefronts from one exclusive scan of the per-wavefront totals.
  constexpr int NW = NT / kWave;
  constexpr int kUnroll = 8;
  const int lane = tid & 63, wave = tid >> 6;
  const int seg = ((n + NW - 1) / NW + 63) & ~63;
  const int w0 = min(n, wave * seg), w1 = min(n, w0 + seg);
  const int sh = 32 - pbits;
  int cgt = 0, ceq = 0;
  for (int b = w0; b < w1; b += 64 * kUnroll) {
    float v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int i = b + u * 64 + lane;
      v[u] = i < w1 ? s[i] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int i = b + u * 64 + lane;
      const uint32_t key = shr32(fkey(v[u]), sh);
      const bool in = i < w1;
      cgt += __popcll(__ballot(in && (all || key > prefix)));
      ceq += __popcll(__ballot(in && !all && key == prefix));
    }
  }
  if (lane == 0) {
    sm[2 * wave] = cgt;
    sm[2 * wave + 1] = ceq;
  }
  __syncthreads();
  int rg = 0, re = 0, tgt = 0, teq = 0;
  for (int w = 0; w < NW; ++w) {
    if (w < wave) {
      rg += sm[2 * w];
      re += sm[2 * w + 1];
    }
    tgt += sm[2 * w];
    teq += sm[2 * w + 1];
  }
  const int total = tgt + min(teq, eq_take);
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int b = w0; b < w1; b += 64 * kUnroll) {
    float v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int i = b + u * 64 + lane;
      v[u] = i < w1 ? s[i] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int i = b + u * 64 + lane;
      const uint32_t key = shr32(fkey(v[u]), sh);
      const bool in = i < w1;
      const bool gt = in && (all || key > prefix);
      const bool eq = in && !all && key == prefix;
      const uint64_t bg = __ballot(gt), be = __ballot(eq);
      const int pg = rg + __popcll(bg & below);
      const int pe = re + __popcll(be & below);
      if (gt || (eq && pe < eq_take)) {
        const int p = pg + min(pe, eq_take);
        if (p < cap) {
          out[p] = i;
          if (out2) out2[p] = i;
        }
      }
      rg += __popcll(bg);
      re += __popcll(be);
    }
  }
  if (tid == 0 && count_out) *count_out = total;
  __syncthreads();
}

// The same selection with every key held in registers. Wavefront w owns the
// contiguous segment [w*64*IPT, (w+1)*64*IPT); within it lane l holds, for each
// group g < IPT/4, the four keys at w*64*IPT + 256*g + 4*l + (0..3), so every load
// instruction reads 1 KB of consecutive scores. Index order inside a segment is
// (group, lane, element). All radix passes and the ordered compaction run on-chip:
// ranks come from ballot popcounts per group plus the per-wavefront totals; no
// further memory round trips. Requires n <= NT * IPT.
//
// Slots past n hold key 0, which no real score produces (every finite or infinite
// float maps above 2^22), so they fall in the lowest histogram bin, never match a
// selected prefix, and need no separate validity test (k >= n, where every score
// is taken, writes 0..n-1 directly). The selection boundary is re-read from LDS,
// wavefront-uniform, before the write walk, so the compiler recomputes the per-key
// predicates instead of keeping them live across the scans.
template <int NT, int IPT, bool OVERLAP = true>
__device__ void wg_select_reg(const float* __restrict__ s, int n, int mode, int k, float thresh,
                              int32_t* __restrict__ out, int cap, int32_t* __restrict__ count_out,
                              int32_t* __restrict__ out2, uint32_t* hist, int* sm) {
  static_assert(IPT % 4 == 0, "IPT must be a multiple of 4");
  constexpr int NW = NT / kWave;
  constexpr int G = IPT / 4;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wbase = wave * 64 * IPT + 4 * lane;     // index of (g = 0, e = 0) for this lane
  const bool vec = (reinterpret_cast<uintptr_t>(s) & 15u) == 0;
  // Top-k that needs the radix passes: with OVERLAP, the first histogram is cleared
  // before the score loads and, when every load can be issued unconditionally
  // (16-byte aligned scores, n a multiple of 4), filled group by group as the loads
  // land (a selection on the critical path: 20.2 -> 16.5 us for 2457 of 49152).
  // Hosted in another kernel's launch it runs off the critical path, and there the
  // plain order measured faster for the host kernel.
  const bool radix = mode != DV_SELECT_THRESHOLD && k > 0 && k < n;
  const bool flat = OVERLAP && vec && (n & 3) == 0 && n >= 4;
  if (radix && OVERLAP) {
    for (int i = tid; i < kSelBins; i += NT) hist[i] = 0u;
    __syncthreads();
  }
  uint32_t key[IPT];
  if (flat) {
    // a group past n re-reads the last four scores (no predicated load, so each
    // group's use waits only for its own load) and gets key 0
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int i = wbase + 256 * g;
      const f32x4 v = *reinterpret_cast<const f32x4*>(s + min(i, n - 4));
#pragma unroll
      for (int e = 0; e < 4; ++e) key[4 * g + e] = i < n ? fkey(v[e]) : 0u;
    }
    if (radix) {
#pragma unroll
      for (int j = 0; j < IPT; ++j) atomicAdd(&hist[key[j] >> (32 - 13)], 1u);
    }
  } else {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int i = wbase + 256 * g;
      if (vec && i + 3 < n) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(s + i);
        key[4 * g] = fkey(v[0]);
        key[4 * g + 1] = fkey(v[1]);
        key[4 * g + 2] = fkey(v[2]);
        key[4 * g + 3] = fkey(v[3]);
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) key[4 * g + e] = i + e < n ? fkey(s[i + e]) : 0u;
      }
    }
  }
  uint32_t prefix = 0u;
  int pbits = 0;
  int eq_take = INT_MAX;
  if (mode == DV_SELECT_THRESHOLD) {
    prefix = fkey(thresh);
    pbits = 32;
  } else if (k >= n) {
    // every score, in index order (the padding slots' keys must not be counted)
    const int m = min(n, cap);
    for (int p = tid; p < m; p += NT) {
      out[p] = p;
      if (out2) out2[p] = p;
    }
    if (tid == 0 && count_out) *count_out = n;
    __syncthreads();
    return;
  } else if (k <= 0) {
    if (tid == 0 && count_out) *count_out = 0;
    __syncthreads();
    return;
  } else {
    int krem = k;
    for (int p = 0; p < 3; ++p) {
      const int D = p < 2 ? 13 : 6, nb = 1 << D;   // 13 + 13 + 6 = 32 key bits
      if (p > 0 || !flat) {
        if (p > 0 || !OVERLAP) {
          for (int i = tid; i < nb; i += NT) hist[i] = 0u;
          __syncthreads();
        }
        const int lo = 32 - pbits - D;
        const int hi = 32 - pbits;
#pragma unroll
        for (int j = 0; j < IPT; ++j) {
          if (shr32(key[j], hi) == prefix) atomicAdd(&hist[(key[j] >> lo) & (uint32_t)(nb - 1)], 1u);
        }
      }
      __syncthreads();
      int dig, above;
      find_digit<NT>(hist, nb, krem, sm, &dig, &above);
      const int cnt = (int)hist[dig];
      krem -= above;
      prefix = (prefix << D) | (uint32_t)dig;
      pbits += D;
      __syncthreads();
      if (cnt == krem) {
        eq_take = INT_MAX;
        break;
      }
      eq_take = krem;
    }
  }
  volatile int* bound = sm + 2 * NW + 4;   // prefix, shift
  if (tid == 0) {
    bound[0] = (int)prefix;
    bound[1] = 32 - pbits;
  }
  // A key is selected when its top pbits bits (13, 26 or 32 here, so the shift is
  // below 32) exceed the prefix; of the keys equal to it, all are taken when eq_take
  // is unbounded (threshold mode, or the last digit's bin was consumed exactly: the
  // usual case, which needs one predicate per key), else the eq_take lowest-indexed.
  // Per-wavefront totals from ballots (no cross-lane shuffles).
  const bool all_eq = eq_take == INT_MAX;
  int sh = 32 - pbits;
  int ngt = 0, neq = 0;
  if (all_eq) {
#pragma unroll
    for (int j = 0; j < IPT; ++j) ngt += __popcll(__ballot((key[j] >> sh) >= prefix));
  } else {
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
      const uint32_t u = key[j] >> sh;
      ngt += __popcll(__ballot(u > prefix));
      neq += __popcll(__ballot(u == prefix));
    }
  }
  if (lane == 0) {
    sm[2 * wave] = ngt;
    sm[2 * wave + 1] = neq;
  }
  __syncthreads();
  int rg = 0, re = 0, tgt = 0, teq = 0;
  for (int w = 0; w < NW; ++w) {
    const int a = sm[2 * w], b = sm[2 * w + 1];
    if (w < wave) {
      rg += a;
      re += b;
    }
    tgt += a;
    teq += b;
  }
  const int total = tgt + min(teq, eq_take);
  prefix = (uint32_t)__builtin_amdgcn_readfirstlane(bound[0]);
  sh = __builtin_amdgcn_readfirstlane(bound[1]);
  // Write walk: group by group; inside a group, lanes in order, then elements. The
  // rank of (lane l, element e) within the group is the number of selected elements
  // of lanes below l (mbcnt over the group's ballots) plus those of lane l before e.
  // put(p, i, take) is called for every slot and stores index i at rank p if take.
  auto below = [](uint64_t m, int acc) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, (uint32_t)acc));
  };
  auto walk_all = [&](auto put) {   // all_eq: one predicate, one running rank
    int r = rg;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      bool sl[4];
      int bl = 0, t = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        sl[e] = (key[4 * g + e] >> sh) >= prefix;
        const uint64_t ms = __ballot(sl[e]);
        bl = below(ms, bl);
        t += __popcll(ms);
      }
      int p = r + bl;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        put(p, wbase + 256 * g + e, sl[e] && p < cap);
        p += sl[e];
      }
      r += t;
    }
  };
  auto walk_ties = [&](auto put) {  // above the prefix, plus the first eq_take equal keys
    int r_gt = rg, r_eq = re;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      bool gt[4], eq[4];
      int bgt = 0, beq = 0, tg = 0, te = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t u = key[4 * g + e] >> sh;
        gt[e] = u > prefix;
        eq[e] = u == prefix;
        const uint64_t mg = __ballot(gt[e]), me = __ballot(eq[e]);
        bgt = below(mg, bgt);
        beq = below(me, beq);
        tg += __popcll(mg);
        te += __popcll(me);
      }
      int pg = r_gt + bgt, pe = r_eq + beq;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int p = pg + min(pe, eq_take);
        put(p, wbase + 256 * g + e, (gt[e] || (eq[e] && pe < eq_take)) && p < cap);
        pg += gt[e];
        pe += eq[e];
      }
      r_gt += tg;
      r_eq += te;
    }
  };
  // A set that fits the histogram's LDS (less 64 slots that take the unselected lanes'
  // writes, so the walk needs no branch) is placed there first and then copied out in
  // contiguous runs; a larger one (threshold mode) is written directly.
  const int m = min(total, cap);
  if (m <= kSelBins - kWave) {
    const int dummy = kSelBins - kWave + lane;
    auto put = [&](int p, int i, bool take) { hist[take ? p : dummy] = (uint32_t)i; };
    if (all_eq)
      walk_all(put);
    else
      walk_ties(put);
    __syncthreads();
    for (int p = tid; p < m; p += NT) {
      const int32_t i = (int32_t)hist[p];
      out[p] = i;
      if (out2) out2[p] = i;
    }
  } else {
    walk_ties([&](int p, int i, bool take) {
      if (take) {
        out[p] = i;
        if (out2) out2[p] = i;
      }
    });
  }
  if (tid == 0 && count_out) *count_out = total;
  __syncthreads();
}

// Selection from a short score vector (n <= NT, one score per thread): the keys are
// staged in LDS and each thread ranks its own against all of them (O(n^2) LDS reads,
// no histogram passes). Same result as wg_select_reg: top-k keeps the k highest keys,
// ties to the lower index (k >= n: every key), threshold keeps every key >= the
// threshold's; the set is written ascending (its first cap members), *count_out gets
// its full size. keys: n u32 of LDS; red: block_excl_scan scratch. Ends with a barrier.
template <int NT>
__device__ void wg_select_small(const float* __restrict__ s, int n, int mode, int k, float thresh,
                                int32_t* __restrict__ out, int cap, int32_t* __restrict__ count_out,
                                int32_t* __restrict__ out2, uint32_t* keys, int* red) {
  const int i = threadIdx.x;
  const uint32_t ki = i < n ? fkey(s[i]) : 0u;
  if (i < n) keys[i] = ki;
  __syncthreads();
  bool sel = false;
  if (i < n) {
    if (mode == DV_SELECT_THRESHOLD) {
      sel = ki >= fkey(thresh);
    } else if (k >= n) {
      sel = true;             // every score
    } else if (k > 0) {
      int rank = 0;
      for (int j = 0; j < n; ++j) {
        const uint32_t kj = keys[j];
        rank += (kj > ki) || (kj == ki && j < i);
      }
      sel = rank < k;
    }
  }
  int total = 0;
  const int p = block_excl_scan<NT>(sel ? 1 : 0, red, &total);
  if (sel && p < cap) {
    out[p] = i;
    if (out2) out2[p] = i;
  }
  if (i == 0 && count_out) *count_out = total;
  __syncthreads();
}

// Top-k selection run by one extra workgroup of another kernel's launch (which leaves
// CUs free for it), so that the selection runs beside that kernel's weight stream
// instead of on the critical path. Inlined: as a call it needs a stack frame for the
// callee-saved registers besides its own spills, which raised the host kernel's
// private segment to 336 bytes per lane and its duration by 1.5-2 us on the
// 3 x 4096-row QKV launch (inlined: 120 bytes).
// Up to 48 * NT scores are selected from registers, larger score vectors stream from
// memory. smem: kSelBins u32 plus kSelSm(NT) ints of LDS.
constexpr int kSelIPT = 48;

template <int NT>
__device__ __forceinline__ void hosted_select(const float* scores, int n, int k, int32_t* idx,
                                              int32_t* idx_out, float* smem) {
  uint32_t* hist = reinterpret_cast<uint32_t*>(smem);
  int* sm = reinterpret_cast<int*>(smem + kSelBins);
  if (n <= NT * kSelIPT)
    wg_select_reg<NT, kSelIPT, false>(scores, n, DV_SELECT_TOPK, k, 0.f, idx, k, nullptr, idx_out, hist, sm);
  else
    wg_select<NT>(scores, n, DV_SELECT_TOPK, k, 0.f, idx, k, nullptr, idx_out, hist, sm);
}

// Top-k of a short score vector (n <= NT) by rank counting; writes the ascending set
// to lds_set[0..k). The keys are staged in LDS first (one coalesced load each), then
// every thread ranks its key against all of them: O(n^2) LDS compares, used for the
// head selection inside other kernels. keys: n u32 of LDS; sel: n ints of LDS.
// Ends with a barrier.
template <int NT>
__device__ void wg_topk_small(const float* __restrict__ s, int n, int k, uint32_t* keys, int* sel,
                              int32_t* lds_set) {
  const int i = threadIdx.x;
  if (i < n) keys[i] = fkey(s[i]);
  __syncthreads();
  if (i < n) {
    const uint32_t ki = keys[i];
    int rank = 0;
    for (int j = 0; j < n; ++j) {
      const uint32_t kj = keys[j];
      rank += (kj > ki) || (kj == ki && j < i);
    }
    sel[i] = rank < k;
  }
  __syncthreads();
  if (i < n && sel[i]) {
    int p = 0;
    for (int j = 0; j < i; ++j) p += sel[j];
    lds_set[p] = i;
  }
  __syncthreads();
}

}  // namespace dv
