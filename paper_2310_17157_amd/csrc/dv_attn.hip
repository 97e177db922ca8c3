// Sparsified multi-head attention (Eq. (2), Section 2.3) at decode time, with the
// KV-cache rule of Section 4.2 (keys and values are computed and stored only for the
// selected heads).
//
//   k_qkv   gathered row-dots: for every selected head i, the dh rows of W^Q_i, W^K_i
//           and W^V_i (contiguous row blocks) against the staged x-hat; q goes to the
//           workspace, k and v to cache row pos. An extra workgroup may host the
//           neuron top-k of the look-ahead layer, or the listing of the selected
//           heads' missing positions for the fill.
//   k_attn  split-KV decode attention: one workgroup per (sequence, selected head,
//           position chunk) computes the chunk's max logit, sum of exponentials and
//           unnormalised value sum; the out-projection kernel combines the chunks.
//   k_kv_fill_listed / k_kv_fill  the missing keys and values of the selected heads
//           (Section 4.2), computed from the kept attention inputs.
#include <math.h>

#include "dv_internal.hpp"
#include "dv_rowdot.hpp"
#include "dv_select.hpp"

namespace dv {

// ------------------------------------------------ missing positions of a head (Section 4.2)
// Threads per listing and positions each thread takes per round.
constexpr int kFillNT = 256, kFillPre = 8;

// The positions below pos whose mark in vh is 0, in ascending order, into out[0..m)
// (when write); returns m. kFillNT threads of the workgroup (lt: their index among
// them) take kFillPre consecutive positions each per round, and a prefix sum over them
// places the positions (wtot: kFillNT / kWave ints of LDS). It holds workgroup barriers:
// every thread of the workgroup calls it, the same number of times.
__device__ __forceinline__ int list_missing(const uint8_t* vh, int pos, int* out, int* wtot, int lt, bool write) {
  constexpr int NW = kFillNT / kWave;
  const int wave = lt >> 6, lane = lt & 63;
  int m = 0;
  for (int c0 = 0; c0 < pos; c0 += kFillNT * kFillPre) {
    const int tb = c0 + lt * kFillPre;
    uint8_t mk[kFillPre];
#pragma unroll
    for (int k = 0; k < kFillPre; ++k) mk[k] = vh[min(tb + k, pos - 1)];
    int cnt = 0;
#pragma unroll
    for (int k = 0; k < kFillPre; ++k) cnt += (tb + k < pos && mk[k] == 0) ? 1 : 0;
    int incl = cnt;                                   // inclusive scan within the wavefront
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int v = __shfl_up(incl, o, kWave);
      if (lane >= o) incl += v;
    }
    if (lane == kWave - 1) wtot[wave] = incl;
    __syncthreads();
    int off = m + incl - cnt, tot = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      off += w < wave ? wtot[w] : 0;
      tot += wtot[w];
    }
    if (write) {
#pragma unroll
      for (int k = 0; k < kFillPre; ++k)
        if (tb + k < pos && mk[k] == 0) out[off++] = tb + k;
    }
    m += tot;
    __syncthreads();                                  // wtot is rewritten by the next round
  }
  return m;
}

// The listing for the missing-KV fill hosted beside the QKV stream by one workgroup of
// NT threads: its NT / kFillNT parts list one selected head each per round.
template <int NT>
__device__ __forceinline__ void hosted_list(const QkvArgs& a) {
  constexpr int NQ = NT / kFillNT;
  __shared__ int wtot[NT / kWave];
  const int qp = (int)threadIdx.x / kFillNT, lt = (int)threadIdx.x - qp * kFillNT;
  for (int j0 = 0; j0 < a.n_heads; j0 += NQ) {
    const int j = j0 + qp, jj = min(j, a.n_heads - 1);
    const int head = min(max(a.heads_in[jj], 0), a.H - 1);
    const int m = list_missing(a.valid + (size_t)head * a.cap, a.pos, a.list + (size_t)jj * a.list_stride,
                               wtot + qp * (kFillNT / kWave), lt, j < a.n_heads);
    if (j < a.n_heads && lt == 0) a.list_count[j] = m;
  }
}

template <typename T, typename KT, int NW, int U, int KX, bool LN>
__global__ void __launch_bounds__(NW * 64) k_qkv(QkvArgs a) {
  extern __shared__ float smem[];
  constexpr int NT = NW * 64;
  const bool host = a.sel_n > 0 || a.list != nullptr;
  const int wg = blockIdx.x, nwg = gridDim.x - (host ? 1 : 0);
  clear_counters(a.clear, a.clear_n);
  if (host && wg == nwg) {
    if (a.sel_n > 0)
      hosted_select<NT>(a.sel_scores, a.sel_n, a.sel_k, a.sel_idx, a.sel_idx_out, smem);
    else
      hosted_list<NT>(a);
    return;
  }
  float* xs = smem;
  float* red = smem + a.d;
  int32_t* hset = reinterpret_cast<int32_t*>(red + NW);
  float* part = reinterpret_cast<float*>(hset + a.n_heads);     // row-dot records
  for (int i = threadIdx.x; i < a.n_heads; i += NT) hset[i] = min(max(a.heads_in[i], 0), a.H - 1);
  __syncthreads();
  if (wg == 0 && a.heads_ws != nullptr)
    for (int i = threadIdx.x; i < a.n_heads; i += NT) a.heads_ws[i] = hset[i];
  if (wg == 0 && a.valid != nullptr)
    for (int h = threadIdx.x; h < a.H; h += NT) {
      uint8_t in = 0;
      for (int i = 0; i < a.n_heads; ++i) in |= hset[i] == h;
      a.valid[(size_t)h * a.cap + a.pos] = in;
    }
  const int per_mat = a.n_heads * a.dh, nqkv = 3 * per_mat;
  auto row_ptr = [&](int row) {
    if (row >= nqkv) {   // appended predictor rows
      const int p = row - nqkv;
      return p < a.r0 ? static_cast<const T*>(a.AT0) + (size_t)p * a.d
                      : static_cast<const T*>(a.AT1) + (size_t)(p - a.r0) * a.d;
    }
    const int m = row / per_mat;
    const int rem = row - m * per_mat;
    const int j = rem / a.dh, t = rem - j * a.dh;
    const void* W = m == 0 ? a.Wq : (m == 1 ? a.Wk : a.Wv);
    return static_cast<const T*>(W) + ((size_t)hset[j] * a.dh + t) * a.d;
  };
  auto epi = [&](int row, float v) {
    if (row >= nqkv) {
      const int p = row - nqkv;
      if (p < a.r0)
        a.hid0[p] = v;
      else
        a.hid1[p - a.r0] = v;
      return;
    }
    const int m = row / per_mat;
    const int rem = row - m * per_mat;
    const int j = rem / a.dh, t = rem - j * a.dh;
    const int head = hset[j];
    const size_t wrow = (size_t)head * a.dh + t;
    const float* bias = m == 0 ? a.bq : (m == 1 ? a.bk : a.bv);
    if (bias) v += bias[wrow];
    if (m == 0) {
      a.q[rem] = v;
    } else {
      KT* C = static_cast<KT*>(m == 1 ? a.K : a.V);
      C[((size_t)head * a.cap + a.pos) * a.dh + t] = (KT)v;
    }
  };
  rowdot_flat<T, NW, U, KX, LN>(row_ptr, epi, nqkv + a.r0 + a.r1, a.d, a.x, a.g, a.be, a.eps, xs, red, part, nullptr,
                                wg, nwg);
}

// CUs left without a QKV workgroup when a selection is hosted in the launch.
constexpr int kQkvSelFreeCUs = 4;

template <typename T, typename KT, int KX>
static hipError_t launch_qkv_t(const QkvArgs& a, hipStream_t st) {
  // 2 loads per batch, two batches in flight per wavefront (measured fastest; 1 and 3
  // were close, 4, 6, 8 and 16 slower): deeper queues only let the XCDs that win the
  // fabric arbitration race ahead of the others
  constexpr int NW = 16, U = 2;
  constexpr int NT = NW * 64;
  const int nrows = 3 * a.n_heads * a.dh + a.r0 + a.r1;
  // One workgroup per CU, each a contiguous range of rows (rowdot_flat). A hosted
  // selection gets one more workgroup, and a few CUs are left free for it to start at once.
  const int cus = device_cu_count();
  const bool host = a.sel_n > 0 || a.list != nullptr;
  const int blocks = max(1, min(nrows, host ? max(1, cus - kQkvSelFreeCUs) : cus));
  size_t lds = (size_t)(a.d + NW) * sizeof(float) + (size_t)a.n_heads * sizeof(int32_t) +
               (size_t)rowdot_flat_part(nrows, blocks, NW) * sizeof(float) + 16;
  if (a.sel_n > 0) lds = max(lds, (size_t)kSelBins * 4 + kSelSm(NT) * sizeof(int));
  const dim3 grid(blocks + (host ? 1 : 0));
  if (a.g != nullptr) {
    const hipError_t e = ensure_dyn_lds(reinterpret_cast<const void*>(k_qkv<T, KT, NW, U, KX, true>), lds);
    if (e != hipSuccess) return e;
    launch_k((k_qkv<T, KT, NW, U, KX, true>), grid, dim3(NW * 64), lds, st, a);
  } else {
    const hipError_t e = ensure_dyn_lds(reinterpret_cast<const void*>(k_qkv<T, KT, NW, U, KX, false>), lds);
    if (e != hipSuccess) return e;
    launch_k((k_qkv<T, KT, NW, U, KX, false>), grid, dim3(NW * 64), lds, st, a);
  }
  return hipGetLastError();
}

template <typename T, typename KT>
static hipError_t launch_qkv_k(const QkvArgs& a, hipStream_t st) {
  switch (rowdot_kx(a.d, 16)) {
    case 1: return launch_qkv_t<T, KT, 1>(a, st);
    case 2: return launch_qkv_t<T, KT, 2>(a, st);
    case 3: return launch_qkv_t<T, KT, 3>(a, st);
    default: return launch_qkv_t<T, KT, 4>(a, st);
  }
}

hipError_t launch_qkv(int wtype, int kvtype, const QkvArgs& a, hipStream_t st) {
  if (wtype == DV_F16)
    return kvtype == DV_F16 ? launch_qkv_k<_Float16, _Float16>(a, st) : launch_qkv_k<_Float16, float>(a, st);
  return kvtype == DV_F16 ? launch_qkv_k<float, _Float16>(a, st) : launch_qkv_k<float, float>(a, st);
}

// ------------------------------------------------------------ attention
// LPP lanes hold one cache row (dh elements, 16 bytes per lane); a wavefront covers
// 64 / LPP positions per step and NSTEP steps per sub-chunk; NW wavefronts per
// workgroup. A workgroup walks its chunk of positions sub-chunk by sub-chunk with a
// running max, sum of exponentials and value sum per wavefront (online softmax), so a
// chunk may be any multiple of the sub-chunk length. The keys and values of the next
// sub-chunk are loaded (two register sets) before the current one is used; loads are
// never predicated (positions past the chunk read its last row and score -inf, lanes
// past the head width read the row's last 16 bytes and are not written out), so the
// waits count exactly the loads of the sub-chunk being used. Keys and values are read
// with non-temporal loads, like the weight streams (at batch 32, 675 MB of them per
// step: 137 -> 110 us against ordinary loads; at batch 1 the two are even).
template <typename KT, int LPP, int NSTEP>
__global__ void __launch_bounds__(256) k_attn(AttnArgs a) {
  constexpr int NW = 4;
  constexpr int E = Chunk<KT>::E;
  constexpr int PPW = 64 / LPP;
  constexpr int SUB = NSTEP * NW * PPW;
  __shared__ float sm_m[NW], sm_l[NW];
  __shared__ float sm_o[NW][256];
  const int j = blockIdx.y, c = blockIdx.x, b = a.reorder ? a.seq_of[blockIdx.z] : (int)blockIdx.z;
  const int jb = b * a.n_heads + j;               // (sequence, selected head)
  const int head = min(max(a.heads[jb], 0), a.H - 1);
  const int t0 = c * a.chunk;
  const int tend = min(t0 + a.chunk, a.posb[b] + 1);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int grp = lane / LPP, gl = lane % LPP;
  const int nchr = a.dh / E;
  const bool lane_on = gl < nchr;
  float qv[E];
#pragma unroll
  for (int e = 0; e < E; ++e) qv[e] = lane_on ? a.q[(size_t)jb * a.dh + gl * E + e] : 0.f;
  const size_t rowb = (size_t)a.dh * sizeof(KT);
  const size_t hoff = ((size_t)b * a.H + head) * a.cap * rowb + (size_t)min(gl, nchr - 1) * 16;
  const char* Kb = static_cast<const char*>(a.K) + hoff;
  const char* Vb = static_cast<const char*>(a.V) + hoff;

  if (a.valid != nullptr)   // every row this workgroup attends holds its key and value
    for (int t = t0 + (int)threadIdx.x; t < tend; t += 256) a.valid[((size_t)b * a.H + head) * a.cap + t] = 1;
  float m = -INFINITY, l = 0.f;
  float o[E];
#pragma unroll
  for (int e = 0; e < E; ++e) o[e] = 0.f;
  auto ldkv = [&](u32x4 (&kw)[NSTEP], u32x4 (&vw)[NSTEP], int sb) {
#pragma unroll
    for (int s = 0; s < NSTEP; ++s) {
      const int t = max(min(sb + (s * NW + wave) * PPW + grp, tend - 1), 0);
      kw[s] = ld_stream(Kb + (size_t)t * rowb);
    }
#pragma unroll
    for (int s = 0; s < NSTEP; ++s) {
      const int t = max(min(sb + (s * NW + wave) * PPW + grp, tend - 1), 0);
      vw[s] = ld_stream(Vb + (size_t)t * rowb);
    }
  };
  auto use = [&](const u32x4 (&kw)[NSTEP], const u32x4 (&vw)[NSTEP], int sb) {
    float sc[NSTEP];
    float mb = -INFINITY;
#pragma unroll
    for (int s = 0; s < NSTEP; ++s) {
      float kv[E];
      unpack<KT>(kw[s], kv);
      float p = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) p = fmaf(qv[e], kv[e], p);
#pragma unroll
      for (int off = LPP / 2; off > 0; off >>= 1) p += __shfl_xor(p, off, kWave);
      const int t = sb + (s * NW + wave) * PPW + grp;
      sc[s] = t < tend ? p * a.scale : -INFINITY;
      mb = fmaxf(mb, sc[s]);
    }
#pragma unroll
    for (int off = LPP; off < 64; off <<= 1) mb = fmaxf(mb, __shfl_xor(mb, off, kWave));
    const float mn = fmaxf(m, mb);
    if (mn != -INFINITY) {
      const float r = m == -INFINITY ? 0.f : __expf(m - mn);
      l *= r;
#pragma unroll
      for (int e = 0; e < E; ++e) o[e] *= r;
#pragma unroll
      for (int s = 0; s < NSTEP; ++s) {
        const float p = sc[s] == -INFINITY ? 0.f : __expf(sc[s] - mn);
        l += p;
        float vv[E];
        unpack<KT>(vw[s], vv);
#pragma unroll
        for (int e = 0; e < E; ++e) o[e] = fmaf(p, vv[e], o[e]);
      }
      m = mn;
    }
  };
  u32x4 ka[NSTEP], va[NSTEP], kb[NSTEP], vb[NSTEP];
  ldkv(ka, va, t0);
  for (int sb = t0; sb < tend;) {
    ldkv(kb, vb, sb + SUB);
    use(ka, va, sb);
    sb += SUB;
    if (sb >= tend) break;
    ldkv(ka, va, sb + SUB);
    use(kb, vb, sb);
    sb += SUB;
  }
  // Each lane's l and o cover its own position group; sum over the groups.
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
  if (a.C != nullptr) {
    // one chunk: H_h(x_b)[t] = o[t] / L, as fp16 coefficients at h's place in the union
    __shared__ int up;
    if (threadIdx.x == 0) {
      int lo = 0, hi = *a.ucount - 1, pp = -1;
      while (lo <= hi) {
        const int mid = (lo + hi) >> 1;
        const int v = a.ulist[mid];
        if (v == head) { pp = mid; break; }
        if (v < head) lo = mid + 1; else hi = mid - 1;
      }
      up = pp;
    }
    __syncthreads();
    if (up < 0 || M == -INFINITY) return;   // (the matrix was cleared)
    float L = 0.f, f[NW];
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      f[w] = sm_m[w] == -INFINITY ? 0.f : __expf(sm_m[w] - M);
      L += sm_l[w] * f[w];
    }
    const float rl = 1.f / L;
    for (int t = threadIdx.x; t < a.dh; t += 256) {
      float acc = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) acc += sm_o[w][t] * f[w];
      a.C[coef_index(b, up * a.dh + t, a.cnb)] = (_Float16)(acc * rl);
    }
    return;
  }
  float* out = a.part + ((size_t)jb * a.n_split + c) * (a.dh + 2);
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

constexpr int kAttnNStep = 4;

static int attn_lpp(int dh, int kvtype) {
  const int nchr = dh * elem_bytes(kvtype) / 16;
  return nchr <= 16 ? 16 : (nchr <= 32 ? 32 : 64);
}

int attn_chunk(int n_heads, int attended, int dh, int kvtype) {
  // Positions per workgroup: a multiple of the sub-chunk (kAttnNStep steps x 4 wavefronts x
  // positions per step). At most kAttnMaxSplit chunks per head (they are combined in
  // the out-projection's prologue); otherwise aim at about one workgroup per CU.
  const int sub = kAttnNStep * 4 * (64 / attn_lpp(dh, kvtype));
  const int nsub = (attended + sub - 1) / sub;
  const int cus = device_cu_count();
  int per = 1;                                               // sub-chunks per workgroup
  while ((long)n_heads * ((nsub + per - 1) / per) > cus && per < nsub) per *= 2;
  while ((nsub + per - 1) / per > kAttnMaxSplit) ++per;
  return per * sub;
}

template <typename KT, int LPP>
static hipError_t launch_attn_l(const AttnArgs& a, int B, hipStream_t st) {
  dim3 grid(a.n_split, a.n_heads, B);
  launch_k((k_attn<KT, LPP, kAttnNStep>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

template <typename KT>
static hipError_t launch_attn_t(const AttnArgs& a, int B, hipStream_t st) {
  switch (attn_lpp(a.dh, sizeof(KT) == 2 ? DV_F16 : DV_F32)) {
    case 16: return launch_attn_l<KT, 16>(a, B, st);
    case 32: return launch_attn_l<KT, 32>(a, B, st);
    default: return launch_attn_l<KT, 64>(a, B, st);
  }
}

hipError_t launch_attn(int kvtype, const AttnArgs& a, int B, hipStream_t st) {
  return kvtype == DV_F16 ? launch_attn_t<_Float16>(a, B, st) : launch_attn_t<float>(a, B, st);
}

// ------------------------------------------------------------ missing keys and values
// Two forms share the group body (fill_group). The listed form (the default) runs after
// a QKV launch that listed the positions, on a resident grid of work items; the form
// below lists in every workgroup and runs when the lists do not fit the workspace:
// one workgroup of 4 wavefronts per (selected head, block of kFillRows rows of
// [W^K_h; W^V_h], group slice). It lists the head's missing positions (valid == 0 below
// pos); wavefront w then takes RPW of the rows (w mod (kFillRows / RPW)) over one of
// kFillCols parts of the columns and, for groups of MT missing positions, walks them in
// 16-byte chunks: the RPW weight chunks and the MT matching slices of the kept inputs
// (L2 hits: every workgroup of the head reads the same few rows of Y) are loaded
// together, two steps in flight, with indices clamped so that no load is predicated.
// The other parts' sums are added to the first's through LDS, in part order. The
// groups of a head are dealt round-robin to kFillSlices workgroups per row block.
// Nothing is read when nothing is missing.
// A fill has few heads with missing rows (about 21 at the benchmark's 59 rows per
// token), so few wavefronts have work: the column parts multiply them and the bytes in
// flight, the slices keep a head missing many positions from being serial work, and
// the prologue's copy of this token's input and the valid marks are read kFillPre per
// thread before any is used. Over 32 decode steps with about 59 missing rows each:
// 70-71 us per fill with 16 rows over all columns per workgroup and no slices, 55-57 us
// with the slices and that prologue, 51 us with two column parts (four: 64 us, the
// listing repeated by four times the workgroups), 44 us with the kept inputs in fp16;
// the listed form, 37.5-38.3 us.
constexpr int kFillRows = 8, kFillCols = 2, kFillSlices = 4;
// The listed fill: rows per wavefront of a work item (items of 2 * kFillListedRPW rows)
// and workgroups per CU of its resident grid (its launch bound).
constexpr int kFillListedRPW = 2, kFillResident = 5;

typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));

// The kept inputs are stored in the cache's type (fp16 or fp32, like the keys and
// values computed from them): four inputs converted with round-to-nearest-even.
__device__ __forceinline__ void keep4(float* dst, f32x4 v) { *reinterpret_cast<f32x4*>(dst) = v; }
__device__ __forceinline__ void keep4(_Float16* dst, f32x4 v) {
  *reinterpret_cast<f16x4*>(dst) = f16x4{(_Float16)v[0], (_Float16)v[1], (_Float16)v[2], (_Float16)v[3]};
}

// The kept-input slice that meets one 16-byte weight chunk of E elements: 8, 16 or 32
// bytes of one position's row, in the cache's type.
template <typename KT, int E> struct Kept;
template <> struct Kept<float, 8> {
  f32x4 v[2];
  __device__ __forceinline__ void load(const float* p) {
    v[0] = *reinterpret_cast<const f32x4*>(p);
    v[1] = *reinterpret_cast<const f32x4*>(p + 4);
  }
  __device__ __forceinline__ float at(int e) const { return v[e >> 2][e & 3]; }
};
template <> struct Kept<float, 4> {
  f32x4 v;
  __device__ __forceinline__ void load(const float* p) { v = *reinterpret_cast<const f32x4*>(p); }
  __device__ __forceinline__ float at(int e) const { return v[e]; }
};
template <> struct Kept<_Float16, 8> {
  f16x8 v;
  __device__ __forceinline__ void load(const _Float16* p) { v = *reinterpret_cast<const f16x8*>(p); }
  __device__ __forceinline__ float at(int e) const { return (float)v[e]; }
};
template <> struct Kept<_Float16, 4> {
  f16x4 v;
  __device__ __forceinline__ void load(const _Float16* p) { v = *reinterpret_cast<const f16x4*>(p); }
  __device__ __forceinline__ float at(int e) const { return (float)v[e]; }
};

// This token's input kept in the cache's type (Y[pos] = x), by one workgroup of kFillNT.
template <typename KT>
__device__ __forceinline__ void keep_input_wg(const KvFillArgs& a) {
  const int n4 = a.d >> 2;                    // (x, Y 16-byte aligned, d % 4 == 0)
  const f32x4* src = reinterpret_cast<const f32x4*>(a.x);
  KT* dst = static_cast<KT*>(a.Y) + (size_t)a.pos * a.d;
  for (int i0 = threadIdx.x; i0 < n4; i0 += kFillNT * kFillPre) {
    f32x4 v[kFillPre];
#pragma unroll
    for (int k = 0; k < kFillPre; ++k) v[k] = src[min(i0 + kFillNT * k, n4 - 1)];
#pragma unroll
    for (int k = 0; k < kFillPre; ++k)
      if (i0 + kFillNT * k < n4) keep4(dst + 4 * (i0 + kFillNT * k), v[k]);
  }
}

// One group of the fill: the keys and values of head `head` at the missing positions
// plist[t0 .. t0 + MT) (clamped to m) for the block rb of NRW * RPW rows of
// [W^K_h; W^V_h]. Wavefront w takes RPW rows (w mod NRW) over one of kFillCols parts of
// the columns, walking them in 16-byte chunks with the RPW weight chunks and the MT
// matching slices of the kept inputs loaded together, two steps in flight (indices
// clamped, so no load is predicated); the other parts' sums are added to the first's
// through LDS (part: [kFillCols - 1][NRW][RPW][MT] floats), in part order.
template <typename T, typename KT, int RPW, int MT>
__device__ __forceinline__ void fill_group(const KvFillArgs& a, int head, int rb, const int* plist, int t0, int m,
                                           float* part) {
  constexpr int E = Chunk<T>::E;
  constexpr int NW = kFillNT / kWave;
  constexpr int NRW = NW / kFillCols;                // wavefronts per column part
  constexpr int RB = NRW * RPW;                      // rows of the block
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int rw = wave % NRW, cp = wave / NRW;
  auto pidx = [&](int q, int r, int u) { return ((q * NRW + rw) * RPW + r) * MT + u; };
  const int nch = a.d / E, nit = (nch + 63) / 64;
  const int it_b = (int)((long)cp * nit / kFillCols), it_e = (int)((long)(cp + 1) * nit / kFillCols);
  // this wavefront's rows (clamped into the block; duplicates are not written)
  const int r0 = rb * RB + rw * RPW, rend = min(2 * a.dh, (rb + 1) * RB);
  const T* W[RPW];
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    const int rr = min(r0 + r, rend - 1);
    const bool isv = rr >= a.dh;
    W[r] = static_cast<const T*>(isv ? a.Wv : a.Wk) + ((size_t)head * a.dh + (isv ? rr - a.dh : rr)) * a.d;
  }
  int pp[MT];
#pragma unroll
  for (int u = 0; u < MT; ++u) pp[u] = plist[min(t0 + u, m - 1)];
  const KT* Yp[MT];
#pragma unroll
  for (int u = 0; u < MT; ++u) Yp[u] = static_cast<const KT*>(a.Y) + (size_t)pp[u] * a.d;
  float acc[RPW][MT];
#pragma unroll
  for (int r = 0; r < RPW; ++r)
#pragma unroll
    for (int u = 0; u < MT; ++u) acc[r][u] = 0.f;
  struct Step {
    u32x4 w[RPW];
    Kept<KT, E> y[MT];
  };
  auto load = [&](Step& st, int it) {
    const int c = min(it * 64 + lane, nch - 1);
#pragma unroll
    for (int r = 0; r < RPW; ++r) st.w[r] = ld_stream(W[r] + (size_t)c * E);
#pragma unroll
    for (int u = 0; u < MT; ++u) st.y[u].load(Yp[u] + (size_t)c * E);
  };
  auto use = [&](const Step& st, int it) {
    if (it * 64 + lane >= nch) return;
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      float wv[E];
      unpack<T>(st.w[r], wv);
#pragma unroll
      for (int u = 0; u < MT; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e) acc[r][u] = fmaf(wv[e], st.y[u].at(e), acc[r][u]);
    }
  };
  // two steps in flight: the next step's loads go out before this step is used
  if (it_b < it_e) {
    Step sa, sb;
    load(sa, it_b);
    for (int it = it_b; it < it_e;) {
      load(sb, min(it + 1, it_e - 1));
      use(sa, it);
      if (++it >= it_e) break;
      load(sa, min(it + 1, it_e - 1));
      use(sb, it);
      ++it;
    }
  }
  // every part reduces its lanes before the barrier (after it, the first part's
  // reductions would lengthen every group's tail: 53.6-55.1 against 50.9-51.4 us per fill)
#pragma unroll
  for (int r = 0; r < RPW; ++r)
#pragma unroll
    for (int u = 0; u < MT; ++u) {
      acc[r][u] = wave_sum(acc[r][u]);
      if (cp > 0 && lane == 0) part[pidx(cp - 1, r, u)] = acc[r][u];
    }
  __syncthreads();
  if (cp == 0) {
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      const int rr = r0 + r;
      const bool isv = rr >= a.dh;
      const int tr = isv ? rr - a.dh : rr;
      const float* bias = isv ? a.bv : a.bk;
      const float bb = (bias != nullptr && rr < rend) ? bias[(size_t)head * a.dh + tr] : 0.f;
#pragma unroll
      for (int u = 0; u < MT; ++u) {
        float v = acc[r][u];
#pragma unroll
        for (int q = 0; q < kFillCols - 1; ++q) v += part[pidx(q, r, u)];
        if (lane == 0 && rr < rend && t0 + u < m) {
          KT* C = static_cast<KT*>(isv ? a.V : a.K);
          C[((size_t)head * a.cap + pp[u]) * a.dh + tr] = (KT)(v + bb);
        }
      }
    }
  }
  __syncthreads();                                    // part is rewritten by the next group
}

// Without a list buffer: one workgroup per (selected head, block of rows, group slice)
// lists its head's missing positions in LDS itself, the slices dealing the head's
// groups of MT positions round-robin.
template <typename T, typename KT, int RPW, int MT>
__global__ void __launch_bounds__(kFillNT, 3) k_kv_fill(KvFillArgs a) {
  constexpr int NW = kFillNT / kWave;
  constexpr int NRW = NW / kFillCols;
  extern __shared__ int flist[];
  __shared__ int wtot[NW];
  __shared__ float part[(kFillCols - 1) * NRW * RPW * MT];
  const int RB = NRW * RPW;
  const int nrb = (2 * a.dh + RB - 1) / RB;
  const int j = blockIdx.x / nrb, rb = blockIdx.x - j * nrb;
  const int head = min(max(a.heads[j], 0), a.H - 1);
  if (blockIdx.x == 0 && blockIdx.y == 0) keep_input_wg<KT>(a);
  const int m = list_missing(a.valid + (size_t)head * a.cap, a.pos, flist, wtot, (int)threadIdx.x, true);
  for (int t0 = (int)blockIdx.y * MT; t0 < m; t0 += MT * (int)gridDim.y)
    fill_group<T, KT, RPW, MT>(a, head, rb, flist, t0, m, part);
}

// The listed fill (the QKV launch listed each selected head's missing positions in
// list[j * stride ..] and their count in count[j]; workgroup 0 keeps this token's
// input): the work items (head with missing positions, block of NRW * RPW
// rows, group of MT positions) are numbered head by head, and a resident grid deals
// them round-robin, so every CU streams a near-equal share of the weight rows however
// the missing positions fall on the heads (a grid per head and block leaves heads
// without missing positions idle and the rest unevenly placed on the CUs).
template <typename T, typename KT, int RPW, int MT>
__global__ void __launch_bounds__(kFillNT, kFillResident) k_kv_fill_listed(KvFillArgs a, const int32_t* list, int stride,
                                                               const int32_t* count) {
  constexpr int NW = kFillNT / kWave;
  constexpr int NRW = NW / kFillCols;
  extern __shared__ int first[];                       // [n_heads + 1] first item of each head
  __shared__ float part[(kFillCols - 1) * NRW * RPW * MT];
  const int RB = NRW * RPW;
  const int nrb = (2 * a.dh + RB - 1) / RB;
  if (blockIdx.x == 0) keep_input_wg<KT>(a);
  if (threadIdx.x == 0) {
    int n = 0;
    for (int j = 0; j < a.n_heads; ++j) {
      first[j] = n;
      n += (min(max(count[j], 0), a.pos) + MT - 1) / MT * nrb;
    }
    first[a.n_heads] = n;
  }
  __syncthreads();
  const int total = first[a.n_heads];
  int j = 0;
  for (int it = blockIdx.x; it < total; it += gridDim.x) {
    while (first[j + 1] <= it) ++j;                    // items ascend, so j only moves forward
    const int k = it - first[j], g = k / nrb, rb = k - g * nrb;
    const int head = min(max(a.heads[j], 0), a.H - 1);
    const int m = min(max(count[j], 0), a.pos);
    const int* hl = list + (size_t)j * stride;
    // a head's last group may hold fewer than MT positions (most heads miss one or two):
    // it loads only the kept inputs it uses
    const int left = m - g * MT;
    if (left >= 3)
      fill_group<T, KT, RPW, MT>(a, head, rb, hl, g * MT, m, part);
    else if (left == 2)
      fill_group<T, KT, RPW, 2>(a, head, rb, hl, g * MT, m, part);
    else
      fill_group<T, KT, RPW, 1>(a, head, rb, hl, g * MT, m, part);
  }
}

template <typename T, typename KT>
static hipError_t launch_kv_fill_t(const KvFillArgs& a, hipStream_t st) {
  constexpr int RPW = kFillRows / (kFillNT / kWave / kFillCols), MT = 4;
  const int nrb = (2 * a.dh + kFillRows - 1) / kFillRows;
  const size_t lds = (size_t)max(a.pos, 1) * sizeof(int);
  const hipError_t e = ensure_dyn_lds(reinterpret_cast<const void*>(k_kv_fill<T, KT, RPW, MT>), lds);
  if (e != hipSuccess) return e;
  launch_k((k_kv_fill<T, KT, RPW, MT>), dim3(max(1, a.n_heads) * nrb, kFillSlices), dim3(kFillNT), lds, st, a);
  return hipGetLastError();
}

hipError_t launch_kv_fill(int wtype, int kvtype, const KvFillArgs& a, hipStream_t st) {
  if (wtype == DV_F16)
    return kvtype == DV_F16 ? launch_kv_fill_t<_Float16, _Float16>(a, st) : launch_kv_fill_t<_Float16, float>(a, st);
  return kvtype == DV_F16 ? launch_kv_fill_t<float, _Float16>(a, st) : launch_kv_fill_t<float, float>(a, st);
}

template <typename T, typename KT>
static hipError_t launch_kv_fill_listed_t(const KvFillArgs& a, const int32_t* list, int stride, hipStream_t st) {
  constexpr int RPW = kFillListedRPW, MT = 4;
  const int32_t* count = list + (size_t)a.n_heads * stride;
  const size_t lds = (size_t)(a.n_heads + 1) * sizeof(int);
  const hipError_t e = ensure_dyn_lds(reinterpret_cast<const void*>(k_kv_fill_listed<T, KT, RPW, MT>), lds);
  if (e != hipSuccess) return e;
  // resident: kFillResident workgroups per CU (the launch bound) deal the items round-robin
  launch_k((k_kv_fill_listed<T, KT, RPW, MT>), dim3(kFillResident * device_cu_count()), dim3(kFillNT), lds, st, a,
           list, stride, count);
  return hipGetLastError();
}

hipError_t launch_kv_fill_listed(int wtype, int kvtype, const KvFillArgs& a, const int32_t* list, int stride,
                                 hipStream_t st) {
  if (wtype == DV_F16)
    return kvtype == DV_F16 ? launch_kv_fill_listed_t<_Float16, _Float16>(a, list, stride, st)
                            : launch_kv_fill_listed_t<_Float16, float>(a, list, stride, st);
  return kvtype == DV_F16 ? launch_kv_fill_listed_t<float, _Float16>(a, list, stride, st)
                          : launch_kv_fill_listed_t<float, float>(a, list, stride, st);
}

template <typename KT>
__global__ void __launch_bounds__(256) k_keep_input(const float* __restrict__ x, KT* __restrict__ Y, int d) {
  const int i = ((int)blockIdx.x * 256 + (int)threadIdx.x) * 4;
  if (i < d) keep4(Y + i, *reinterpret_cast<const f32x4*>(x + i));
}

hipError_t launch_keep_input(int kvtype, const KvFillArgs& a, hipStream_t st) {
  const dim3 grid((a.d / 4 + 255) / 256);
  if (kvtype == DV_F16)
    launch_k(k_keep_input<_Float16>, grid, dim3(256), 0, st, a.x, static_cast<_Float16*>(a.Y) + (size_t)a.pos * a.d, a.d);
  else
    launch_k(k_keep_input<float>, grid, dim3(256), 0, st, a.x, static_cast<float*>(a.Y) + (size_t)a.pos * a.d, a.d);
  return hipGetLastError();
}

}  // namespace dv
