// Decode-stage kernels: boundary test (Section 4.1), decode store_cache with
// segment eviction (Section 4.2 decode stage), group-consistent retrieval
// (Appendix B; Algorithm 1 Retrieve) and sparse decode attention (Section 3.1).
#include <algorithm>
#include <cstdlib>

#include <mutex>

#include "common.h"

namespace louiskv {
namespace {

constexpr int kMaxGroupSize = 8;
constexpr int kMaxUnits = 8192;

// Per-slice state of a local window with boundary-delimited segments (int32):
// units so far, first token (generation index) in the window, the ring of
// segment first tokens (oldest at head, count entries, the last one open),
// and a flag set when a segment could not become a unit (unit table full).
constexpr int kSegNUnits = 0, kSegWinFirst = 1, kSegHead = 2, kSegCount = 3, kSegOverflow = 4;
constexpr int kSegRing = 8;   // the ring of `window` entries starts here

// ------------------------------------------------------------------ boundary

// Sum over the 16 lanes of a DPP row for a float64 (two 32-bit DPP moves per step).
__device__ __forceinline__ double row16_sum_f64(double x) {
#define LKV_DPP64(ctrl)                                                                                   \
  {                                                                                                       \
    const int lo = __builtin_amdgcn_update_dpp(0, (int)__double2loint(x), ctrl, 0xF, 0xF, false);        \
    const int hi = __builtin_amdgcn_update_dpp(0, (int)__double2hiint(x), ctrl, 0xF, 0xF, false);        \
    x += __hiloint2double(hi, lo);                                                                        \
  }
  LKV_DPP64(0xB1) LKV_DPP64(0x4E) LKV_DPP64(0x141) LKV_DPP64(0x140)
#undef LKV_DPP64
  return x;
}

// Eight consecutive elements of a row as float (16 B of bf16, 32 B of fp32).
__device__ __forceinline__ void load_row8(const uint16_t* p, float* x) {
  const uint4 v = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void load_row8(const float* p, float* x) {
  const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}

constexpr int kBndHeadsPerPass = 32;   // 16 lane groups x 2 heads, all loads issued together

// r of group g (Section 4.1): the mean over the group's n_heads query heads
// of cos(q_ref, q), in float64; NaN at the first step.  Threads 0..255 load:
// 16 lanes per head (lane sub holds dims 8*sub..+7), each 16-lane group takes
// two heads per pass, the dot product and norms of a head are DPP row sums.
// Every thread of the block must call it (one barrier); every thread gets r,
// summed in the same order, so blocks that test the same group agree bit
// for bit.
template <class T>
__device__ __forceinline__ double boundary_r(const T* __restrict__ q, const T* __restrict__ q_ref, int n_heads,
                                             int first, int64_t g, double* s_part /* [16] in LDS */) {
  const int tid = threadIdx.x, sub = tid & 15, hg = tid >> 4;
  const size_t base = (size_t)g * n_heads * kHeadDim;
  double acc = 0.0;
  if (!first && tid < 256) {
    for (int p = 0; p < n_heads; p += kBndHeadsPerPass) {
      float a[2][8], b[2][8];
      bool ok[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int h = p + hg + 16 * i;
        ok[i] = h < n_heads;
        const size_t o = base + (size_t)(ok[i] ? h : 0) * kHeadDim + 8 * sub;
        load_row8(q + o, a[i]);
        load_row8(q_ref + o, b[i]);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        double dot = 0.0, na = 0.0, nb = 0.0;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          dot = fma((double)a[i][e], (double)b[i][e], dot);
          na = fma((double)a[i][e], (double)a[i][e], na);
          nb = fma((double)b[i][e], (double)b[i][e], nb);
        }
        dot = row16_sum_f64(dot);
        na = row16_sum_f64(na);
        nb = row16_sum_f64(nb);
        if (ok[i]) acc += dot / fmax(sqrt(na) * sqrt(nb), 1e-30);
      }
    }
  }
  if (tid < 256 && sub == 0) s_part[hg] = acc;
  __syncthreads();
  if (first) return __builtin_nan("");
  double r = 0.0;
  for (int i = 0; i < 16; ++i) r += s_part[i];
  return r / (double)n_heads;
}

// One block of 4 waves per group: r, the decision (first step, or r < tau),
// and the reference query's update (every step in PREV mode, at a fire in
// ANCHOR mode).
template <class T>
__device__ __forceinline__ void boundary_group(const T* __restrict__ q, T* __restrict__ q_ref, int n_heads,
                                               double tau, int mode, int first, double* __restrict__ r_out,
                                               uint8_t* __restrict__ fire_out, int g) {
  __shared__ double s_part[16];
  const int tid = threadIdx.x;
  const size_t base = (size_t)g * n_heads * kHeadDim;
  const double r = boundary_r(q, q_ref, n_heads, first, g, s_part);
  const int fire = first ? 1 : (r < tau ? 1 : 0);
  if (tid == 0) {
    if (r_out) r_out[g] = r;
    fire_out[g] = (uint8_t)fire;
  }
  __syncthreads();   // every thread has read q_ref before it is rewritten
  if (mode == LOUISKV_REF_PREV || fire) {
    const int n = n_heads * kHeadDim;
    for (int i = tid; i < n; i += 256) q_ref[base + i] = q[base + i];
  }
}

template <class T>
__global__ __launch_bounds__(256)
void boundary_kernel(const T* __restrict__ q, T* __restrict__ q_ref, int n_heads, double tau, int mode,
                     int first, double* __restrict__ r_out, uint8_t* __restrict__ fire_out) {
  boundary_group(q, q_ref, n_heads, tau, mode, first, r_out, fire_out, (int)blockIdx.x);
}

// ------------------------------------------------------------------ decode store

// One wave per slice: optional eviction of the oldest segment (mean key as a new
// unit, rows copied to the pool), then the new token enters its ring slot.
// (Lane l moves dims 2l, 2l+1 of every row, so the eviction's reads of the
// oldest slots and the new token's write into one of them are one lane's
// accesses, in its program order; the wave waits for its loads before the
// write.)
template <class T>
__device__ __forceinline__ void store_slice(const T* __restrict__ k_new, const T* __restrict__ v_new,
                                            T* __restrict__ k_local, T* __restrict__ v_local, int window, int step,
                                            int seg_len, int evict_seg, float* __restrict__ reps,
                                            int32_t* __restrict__ unit_start, int32_t* __restrict__ unit_size,
                                            int units_cap, int n_clusters, T* __restrict__ k_pool,
                                            T* __restrict__ v_pool, int64_t pool_rows, int prompt_len, int64_t s,
                                            int lane) {
  const size_t lbase = (size_t)s * window * kHeadDim;
  if (evict_seg >= 0) {
    const int slot0 = (int)(((int64_t)evict_seg * seg_len) % window);
    const int unit = n_clusters + evict_seg;
    const int64_t prow = (int64_t)prompt_len + (int64_t)evict_seg * seg_len;
    double a0 = 0.0, a1 = 0.0;
    for (int r = 0; r < seg_len; ++r) {
      const size_t o = lbase + (size_t)(slot0 + r) * kHeadDim + 2 * lane;
      const T k0 = k_local[o], k1 = k_local[o + 1];
      a0 += (double)load_as_f32(&k0, 0);
      a1 += (double)load_as_f32(&k1, 0);
      if (k_pool) {
        const size_t po = ((size_t)s * pool_rows + prow + r) * kHeadDim + 2 * lane;
        k_pool[po] = k0;
        k_pool[po + 1] = k1;
        if (v_pool) {
          v_pool[po] = v_local[o];
          v_pool[po + 1] = v_local[o + 1];
        }
      }
    }
    float* rep = reps + ((size_t)s * units_cap + unit) * kHeadDim;
    rep[2 * lane] = (float)(a0 / (double)seg_len);
    rep[2 * lane + 1] = (float)(a1 / (double)seg_len);
    if (lane == 0) {
      unit_start[s * units_cap + unit] = (int32_t)prow;
      unit_size[s * units_cap + unit] = seg_len;
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // the evicted rows are in before the slot is rewritten
  }
  const int slot = step % window;
  const size_t o = lbase + (size_t)slot * kHeadDim + 2 * lane;
  const size_t n = (size_t)s * kHeadDim + 2 * lane;
  k_local[o] = k_new[n];
  k_local[o + 1] = k_new[n + 1];
  v_local[o] = v_new[n];
  v_local[o + 1] = v_new[n + 1];
}

template <class T>
__global__ __launch_bounds__(64)
void store_decode_kernel(const T* __restrict__ k_new, const T* __restrict__ v_new, T* __restrict__ k_local,
                         T* __restrict__ v_local, int window, int step, int seg_len, int evict_seg,
                         float* __restrict__ reps, int32_t* __restrict__ unit_start, int32_t* __restrict__ unit_size,
                         int units_cap, int n_clusters, T* __restrict__ k_pool, T* __restrict__ v_pool,
                         int64_t pool_rows, int prompt_len) {
  store_slice(k_new, v_new, k_local, v_local, window, step, seg_len, evict_seg, reps, unit_start, unit_size,
              units_cap, n_clusters, k_pool, v_pool, pool_rows, prompt_len, (int64_t)blockIdx.x, (int)threadIdx.x);
}

// The boundary test and the fixed-segment store of one decode step in one
// launch: blocks 0..n_groups-1 test their group, the others store four slices
// each (one wave per slice).  The two are independent: the store writes only
// the unit it creates and rows past every existing unit, which this step's
// retrieval does not read.
template <class T>
__global__ __launch_bounds__(256)
void decode_prologue_kernel(const T* __restrict__ q, T* __restrict__ q_ref, int n_heads, double tau, int mode,
                            int first, double* __restrict__ r_out, uint8_t* __restrict__ fire_out, int n_groups,
                            const T* __restrict__ k_new, const T* __restrict__ v_new, T* __restrict__ k_local,
                            T* __restrict__ v_local, int64_t n_slices, int window, int step, int seg_len,
                            int evict_seg, float* __restrict__ reps, int32_t* __restrict__ unit_start,
                            int32_t* __restrict__ unit_size, int units_cap, int n_clusters, T* __restrict__ k_pool,
                            T* __restrict__ v_pool, int64_t pool_rows, int prompt_len) {
  if ((int)blockIdx.x < n_groups) {
    boundary_group(q, q_ref, n_heads, tau, mode, first, r_out, fire_out, (int)blockIdx.x);
    return;
  }
  const int64_t s = (int64_t)(blockIdx.x - n_groups) * 4 + (threadIdx.x >> 6);
  if (s >= n_slices) return;
  store_slice(k_new, v_new, k_local, v_local, window, step, seg_len, evict_seg, reps, unit_start, unit_size,
              units_cap, n_clusters, k_pool, v_pool, pool_rows, prompt_len, s, (int)(threadIdx.x & 63));
}

// store_cache(decode) with boundary-delimited segments, one wave per slice.
// Token `step` opens a new segment when its group fired, when no segment is
// open, or when the open one already holds seg_max tokens.  If the window
// already holds `window` tokens, the oldest segment (closed: seg_max < window)
// leaves first: its mean key (float64 sum, one rounding) becomes unit
// n_units with pool rows prompt_len + its first token .. (tokens leave in
// order, so a token's pool row is prompt_len + its generation index).  Then
// the token goes to ring slot step % window.  The state starts from
// seg_state_init_kernel.
template <class T>
__global__ __launch_bounds__(64)
void store_segmented_kernel(const T* __restrict__ k_new, const T* __restrict__ v_new, T* __restrict__ k_local,
                            T* __restrict__ v_local, int window, int step, int seg_max,
                            const uint8_t* __restrict__ fire, int n_kv_heads, int32_t* __restrict__ state,
                            float* __restrict__ reps, int32_t* __restrict__ unit_start,
                            int32_t* __restrict__ unit_size, int units_cap, int n_clusters, T* __restrict__ k_pool,
                            T* __restrict__ v_pool, int64_t pool_rows, int prompt_len) {
  const int64_t s = blockIdx.x;
  const int lane = threadIdx.x;
  int32_t* st = state + s * (kSegRing + window);
  int32_t* ring = st + kSegRing;
  int n_units = st[kSegNUnits], win_first = st[kSegWinFirst], head = st[kSegHead], count = st[kSegCount],
      overflow = st[kSegOverflow];
  const bool fired = fire && fire[s / n_kv_heads] != 0;
  const int open_first = count > 0 ? ring[(head + count - 1) % window] : -1;
  const bool opens = count == 0 || fired || step - open_first >= seg_max;
  const size_t lbase = (size_t)s * window * kHeadDim;
  if (step - win_first >= window && count > 0) {
    const int a = ring[head];
    const int b = count > 1 ? ring[(head + 1) % window] : step;
    const int len = b - a;
    const int64_t prow = (int64_t)prompt_len + a;
    const bool room = n_units < units_cap && prow + len <= pool_rows;
    double a0 = 0.0, a1 = 0.0;
    for (int r = 0; r < len; ++r) {
      const size_t o = lbase + (size_t)((a + r) % window) * kHeadDim + 2 * lane;
      const T k0 = k_local[o], k1 = k_local[o + 1];
      a0 += (double)load_as_f32(&k0, 0);
      a1 += (double)load_as_f32(&k1, 0);
      if (k_pool && room) {
        const size_t po = ((size_t)s * pool_rows + prow + r) * kHeadDim + 2 * lane;
        k_pool[po] = k0;
        k_pool[po + 1] = k1;
        if (v_pool) {
          v_pool[po] = v_local[o];
          v_pool[po + 1] = v_local[o + 1];
        }
      }
    }
    if (room) {
      float* rep = reps + ((size_t)s * units_cap + n_units) * kHeadDim;
      rep[2 * lane] = (float)(a0 / (double)len);
      rep[2 * lane + 1] = (float)(a1 / (double)len);
      if (lane == 0) {
        unit_start[s * units_cap + n_units] = (int32_t)prow;
        unit_size[s * units_cap + n_units] = len;
      }
      ++n_units;
    } else {
      overflow = 1;   // no room for the unit: its tokens are no longer attended
    }
    head = (head + 1) % window;
    --count;
    win_first = b;
    __syncthreads();   // the evicted rows are read before the new token overwrites the first slot
  }
  if (opens) {
    if (lane == 0) ring[(head + count) % window] = step;
    ++count;
  }
  const int slot = step % window;
  const size_t o = lbase + (size_t)slot * kHeadDim + 2 * lane;
  const size_t n = (size_t)s * kHeadDim + 2 * lane;
  k_local[o] = k_new[n];
  k_local[o + 1] = k_new[n + 1];
  v_local[o] = v_new[n];
  v_local[o + 1] = v_new[n + 1];
  if (lane == 0) {
    st[kSegNUnits] = n_units;
    st[kSegWinFirst] = win_first;
    st[kSegHead] = head;
    st[kSegCount] = count;
    st[kSegOverflow] = overflow;
  }
}

// The state before the first decode step: the clusters are the only units,
// the window is empty.
__global__ void seg_state_init_kernel(int32_t* __restrict__ state, int64_t n_slices, int stride, int n_clusters) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_slices * stride) return;
  const int e = (int)(i % stride);
  state[i] = e == kSegNUnits ? n_clusters : 0;
}

// ------------------------------------------------------------------ retrieve

#ifndef LKV_SEL_THREADS
#define LKV_SEL_THREADS 512
#endif
constexpr int kSelThreads = LKV_SEL_THREADS;
constexpr int kSelWaves = kSelThreads / 64;
// The selection's score sums are taken as kSumThreads threads would take
// them, for every block size that divides it (see select_after_max).
constexpr int kSumThreads = 512;
constexpr int kSmallSelThreads = 256;   // retrieval blocks when slices outnumber compute units
static_assert(kSumThreads % kSelThreads == 0, "the block size must divide the summation width");
constexpr int kUnitIdBits = 13;       // kMaxUnits = 2^13

// Sort key of a unit: larger is ranked first.  The score (a non-negative
// double, whose bit pattern orders like its value) keeps its top 51 bits and
// the low 13 bits hold (kMaxUnits - 1 - id), so equal keys rank the lower id
// first.  Scores closer than 2^-39 relative order by id.
__device__ __forceinline__ uint64_t unit_key(double a, int id) {
  const uint64_t bits = (uint64_t)__double_as_longlong(a);
  return (bits >> kUnitIdBits << kUnitIdBits) | (uint64_t)(kMaxUnits - 1 - id);
}
__device__ __forceinline__ int key_unit(uint64_t k) { return kMaxUnits - 1 - (int)(k & (kMaxUnits - 1)); }

// The key of lane (lane ^ JJ), JJ < 64.  Distances 1 and 2 are quad
// permutations and 4 and 8 row shifts (DPP, no LDS crossbar); 16 and 32 go
// through ds_bpermute.
template <int JJ>
__device__ __forceinline__ uint64_t xor_partner_u64(uint64_t v, int lane) {
  const int lo = (int)(uint32_t)v, hi = (int)(uint32_t)(v >> 32);
  int plo, phi;
  if constexpr (JJ == 1 || JJ == 2) {
    constexpr int ctl = JJ == 1 ? 0xB1 : 0x4E;   // quad_perm [1,0,3,2] and [2,3,0,1]
    plo = __builtin_amdgcn_update_dpp(lo, lo, ctl, 0xF, 0xF, false);
    phi = __builtin_amdgcn_update_dpp(hi, hi, ctl, 0xF, 0xF, false);
  } else if constexpr (JJ == 4 || JJ == 8) {
    // inside a 16-lane row: lanes with bit JJ clear read lane + JJ (row_shl),
    // the others lane - JJ (row_shr)
    const int alo = __builtin_amdgcn_update_dpp(lo, lo, 0x100 + JJ, 0xF, 0xF, false);
    const int ahi = __builtin_amdgcn_update_dpp(hi, hi, 0x100 + JJ, 0xF, 0xF, false);
    const int blo = __builtin_amdgcn_update_dpp(lo, lo, 0x110 + JJ, 0xF, 0xF, false);
    const int bhi = __builtin_amdgcn_update_dpp(hi, hi, 0x110 + JJ, 0xF, 0xF, false);
    const bool up = (lane & JJ) != 0;
    plo = up ? blo : alo;
    phi = up ? bhi : ahi;
  } else {
    plo = __shfl_xor(lo, JJ, kWave);
    phi = __shfl_xor(hi, JJ, kWave);
  }
  return ((uint64_t)(uint32_t)phi << 32) | (uint32_t)plo;
}

// One compare-exchange step at distance JJ of bitonic stage k (element index i).
template <int JJ>
__device__ __forceinline__ uint64_t bitonic_step(uint64_t v, int i, int k) {
  const uint64_t o = xor_partner_u64<JJ>(v, i & 63);
  // the lane keeps the larger key iff its block sorts descending and it is
  // the lower element of the pair, or ascending and the upper one; keys are
  // distinct except padding zeros, so one compare decides
  const bool keep_larger = ((i & k) == 0) == ((i & JJ) == 0);
  return ((v > o) == keep_larger) ? v : o;
}

// Bitonic merge steps jj = jj0, jj0/2, .., 1 of stage k on two independent
// keys per lane (element indices i0, i1 = 64*chunk + lane; partners are in
// the same wave); two chains give the scheduler independent work to overlap.
__device__ __forceinline__ void bitonic_in_wave2(uint64_t& v0, uint64_t& v1, int i0, int i1, int k, int jj0) {
  if (jj0 >= 32) { v0 = bitonic_step<32>(v0, i0, k); v1 = bitonic_step<32>(v1, i1, k); }
  if (jj0 >= 16) { v0 = bitonic_step<16>(v0, i0, k); v1 = bitonic_step<16>(v1, i1, k); }
  if (jj0 >= 8) { v0 = bitonic_step<8>(v0, i0, k); v1 = bitonic_step<8>(v1, i1, k); }
  if (jj0 >= 4) { v0 = bitonic_step<4>(v0, i0, k); v1 = bitonic_step<4>(v1, i1, k); }
  if (jj0 >= 2) { v0 = bitonic_step<2>(v0, i0, k); v1 = bitonic_step<2>(v1, i1, k); }
  v0 = bitonic_step<1>(v0, i0, k);
  v1 = bitonic_step<1>(v1, i1, k);
}

// A wave's 128 keys (two a lane: element indices lane and 64 + lane) sorted
// in descending order, in registers.
__device__ __forceinline__ void sort128_desc(uint64_t& v0, uint64_t& v1, int lane) {
  const int i0 = lane, i1 = kWave + lane;
#pragma unroll
  for (int k = 2; k <= kWave; k <<= 1) bitonic_in_wave2(v0, v1, i0, i1, k, k >> 1);
  // stage 128, distance 64: the partners are a lane's two keys
  if (v0 < v1) {
    const uint64_t t = v0;
    v0 = v1;
    v1 = t;
  }
  bitonic_in_wave2(v0, v1, i0, i1, 2 * kWave, kWave / 2);
}

// The 128 largest of two descending 128-key lists (t, v; same layout), in
// descending order into t: the elementwise maxima of t and v reversed are
// those keys as a bitonic sequence, which the last stage of the network sorts.
__device__ __forceinline__ void merge_top128(uint64_t& t0, uint64_t& t1, uint64_t v0, uint64_t v1, int lane) {
  const int src = kWave - 1 - lane;   // element 127 - i of v sits in lane 63 - i%64, the other register
  const uint64_t r1 = ((uint64_t)(uint32_t)__shfl((int)(uint32_t)(v1 >> 32), src, kWave) << 32) |
                      (uint32_t)__shfl((int)(uint32_t)v1, src, kWave);
  const uint64_t r0 = ((uint64_t)(uint32_t)__shfl((int)(uint32_t)(v0 >> 32), src, kWave) << 32) |
                      (uint32_t)__shfl((int)(uint32_t)v0, src, kWave);
  t0 = t0 > r1 ? t0 : r1;
  t1 = t1 > r0 ? t1 : r0;
  if (t0 < t1) {
    const uint64_t t = t0;
    t0 = t1;
    t1 = t;
  }
  bitonic_in_wave2(t0, t1, lane, kWave + lane, 2 * kWave, kWave / 2);
}

constexpr int kLogitThreads = 256;
constexpr int kLogitWaves = kLogitThreads / 64;
constexpr int kMaxLogitParts = 16;
// Parts of a fused decode step's selection: up to one per block of a slice.
constexpr int kMaxSelectParts = 32;

// Logit workspace per call: the logits [S][units_cap][kMaxGroupSize].
size_t logit_ws_doubles(int64_t S, int units_cap) { return (size_t)S * units_cap * kMaxGroupSize; }

// Unit count of slice ps: the argument, or its own count with
// boundary-delimited segments (the argument then bounds it).
__device__ __forceinline__ int slice_units(const int32_t* seg_state, int seg_stride, int64_t ps, int n_units_arg) {
  return seg_state ? min(max(seg_state[ps * seg_stride + kSegNUnits], 1), n_units_arg) : n_units_arg;
}

// Logits l_ju = q_j . rep_u * scale of the group-consistent score (Appendix
// B) in float64.  A unit's 128 dimensions are split over kLPU lanes (8 for
// up to 4 heads per group, else 16): lane `sub` holds the 4-dim pieces
// 4*sub + 4*kLPU*c (c = 0 .. kDims/4 - 1) of the G queries in float64
// registers, so that each 16-byte load of a lane group reads whole 128-byte
// lines of the unit's row; the lanes' partial dot products are summed over
// the lane group by DPP.  A wave takes 32 units per iteration,
// all their loads in flight (16 KiB a wave).  The per-stage and the fused selection kernels
// share this code, so their scores are equal bit for bit.
template <int G>
struct LogitLayout {
  static constexpr int kLPU = G <= 4 ? 8 : 16;        // lanes per unit
  static constexpr int kDims = kHeadDim / kLPU;       // dims per lane
  static constexpr int kGroups = 64 / kLPU;           // units per wave instruction
  static constexpr int kPerLane = 32 / kGroups;       // units per lane per iteration
};
constexpr int kLogitUnitsPerIter = 32;

template <int G, class T>
__device__ __forceinline__ void load_q_f64(const T* __restrict__ q, size_t row0, int lane,
                                           double (&qd)[G][LogitLayout<G>::kDims]) {
  using LL = LogitLayout<G>;
  const int sub = lane % LL::kLPU;
#pragma unroll
  for (int j = 0; j < G; ++j)
#pragma unroll
    for (int e = 0; e < LL::kDims; ++e)
      qd[j][e] = (double)load_as_f32(q, (row0 + j) * kHeadDim + (e / 4) * (4 * LL::kLPU) + 4 * sub + e % 4);
}

// Sum of a float64 over the kLPU lanes of a unit's lane group.
template <int kLPU>
__device__ __forceinline__ double lane_group_sum_f64(double x) {
#define LKV_DPP64(ctrl)                                                                                   \
  {                                                                                                       \
    const int lo = __builtin_amdgcn_update_dpp(0, (int)__double2loint(x), ctrl, 0xF, 0xF, false);        \
    const int hi = __builtin_amdgcn_update_dpp(0, (int)__double2hiint(x), ctrl, 0xF, 0xF, false);        \
    x += __hiloint2double(hi, lo);                                                                        \
  }
  LKV_DPP64(0xB1) LKV_DPP64(0x4E) LKV_DPP64(0x141)
  if constexpr (kLPU == 16) LKV_DPP64(0x140)
#undef LKV_DPP64
  return x;
}

// The logits of units u0 .. u0 + 31 (those below u_end): maxima per head into
// mx, each logit stored once (kShared: with device-scope stores, for another
// block of the same launch to read).
template <int G, bool kShared>
__device__ __forceinline__ void wave_unit_logits(const double (&qd)[G][LogitLayout<G>::kDims],
                                                 const float* __restrict__ rs, int u0, int u_end, double scale,
                                                 double* __restrict__ lg, double (&mx)[G], int lane) {
  using LL = LogitLayout<G>;
  const int sub = lane % LL::kLPU, gid = lane / LL::kLPU;
  float4 x[LL::kPerLane][LL::kDims / 4];
#pragma unroll
  for (int i = 0; i < LL::kPerLane; ++i) {
    const int u = min(u0 + i * LL::kGroups + gid, u_end - 1);   // past the end: re-read the last unit, unused
    const float* r = rs + (size_t)u * kHeadDim + 4 * sub;
#pragma unroll
    for (int c = 0; c < LL::kDims / 4; ++c) x[i][c] = *reinterpret_cast<const float4*>(r + 4 * LL::kLPU * c);
  }
#pragma unroll
  for (int i = 0; i < LL::kPerLane; ++i) {
    const int u = u0 + i * LL::kGroups + gid;
    double xd[LL::kDims];
#pragma unroll
    for (int c = 0; c < LL::kDims / 4; ++c) {
      xd[4 * c] = x[i][c].x; xd[4 * c + 1] = x[i][c].y; xd[4 * c + 2] = x[i][c].z; xd[4 * c + 3] = x[i][c].w;
    }
#pragma unroll
    for (int j = 0; j < G; ++j) {
      double a = 0.0;
#pragma unroll
      for (int e = 0; e < LL::kDims; ++e) a = fma(qd[j][e], xd[e], a);
      a = lane_group_sum_f64<LL::kLPU>(a) * scale;
      if (u < u_end) {
        mx[j] = fmax(mx[j], a);
        if (sub == j) {
          if constexpr (kShared)
            __hip_atomic_store(lg + (size_t)u * G + j, a, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          else
            lg[(size_t)u * G + j] = a;
        }
      }
    }
  }
}

// The logits of one part of one fired slice's units (n_parts blocks per
// slice, so that few slices still spread over many CUs).
template <class T, int G>
__global__ __launch_bounds__(kLogitThreads)
void unit_logits_kernel(const T* __restrict__ q, int n_kv_heads, double scale, const float* __restrict__ reps,
                        int units_cap, int n_units_arg, const uint8_t* __restrict__ fire,
                        double* __restrict__ logit_ws, const int32_t* __restrict__ seg_state, int seg_stride,
                        int slice_div, int n_parts) {
  const int64_t s = blockIdx.x / n_parts;
  const int part = (int)(blockIdx.x - s * n_parts);
  const int64_t grp = s / n_kv_heads;
  if (fire && !fire[grp]) return;
  const int64_t ps = s / slice_div;     // per-head lists read their KV head's units
  const int n_units = slice_units(seg_state, seg_stride, ps, n_units_arg);
  const int per = (n_units + n_parts - 1) / n_parts;
  const int u_begin = part * per, u_end = min(n_units, u_begin + per);
  if (u_begin >= u_end) return;
  const int kvh = (int)(s - grp * n_kv_heads);
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n_q_heads = n_kv_heads * G;
  double qd[G][LogitLayout<G>::kDims];
  load_q_f64<G>(q, (size_t)grp * n_q_heads + (size_t)kvh * G, lane, qd);
  double* lg = logit_ws + (size_t)s * units_cap * G;
  const float* rs = reps + (size_t)ps * units_cap * kHeadDim;
  double mx[G];   // unused here: the selection kernel takes the maxima of the stored logits
#pragma unroll
  for (int j = 0; j < G; ++j) mx[j] = -__builtin_inf();
  for (int u0 = u_begin + w * kLogitUnitsPerIter; u0 < u_end; u0 += kLogitWaves * kLogitUnitsPerIter)
    wave_unit_logits<G, false>(qd, rs, u0, u_end, scale, lg, mx, lane);
}

// Number of logit blocks per slice: 1 (the selection kernel computes them
// itself) once there are enough slices for the chip, else enough blocks
// for it, at least 64 units per block.
int logit_parts(int64_t n_slices, int n_units) {
  if (n_slices >= 128) return 1;
  int parts = (int)std::min<int64_t>(kMaxLogitParts, std::max<int64_t>(1, (1024 + n_slices - 1) / n_slices));
  while (parts > 1 && (n_units + parts - 1) / parts < 64) --parts;
  return parts;
}

// A logit of the selection workspace.  kShared: written by other blocks of
// the same launch, so read coherently at device scope (the per-XCD L2 may
// hold an older copy of the line).
template <bool kShared>
__device__ __forceinline__ double load_logit(const double* p) {
  if constexpr (kShared)
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else
    return *p;
}

// The selection of one fired slice once its logits l_ju (lg, [unit][G]) and
// their per-head maxima M_j (s_m) are known, with the unit sizes in s_size:
//  pass 2  e_ju = exp(l_ju - M_j) and Z_j = sum_u e_ju (the block's threads);
//  pass 3  A_u = (1/g) sum_j e_ju / Z_j and the sort keys;
//  sort    64-key chunks in registers for merge distances below 64 (no
//          barrier), LDS steps with a barrier for the longer ones;
//  then the prefix stop under the budget, the selected unit list and the
//  pool-row list.  kShared: the logits come from other blocks of the launch;
//  they are read coherently and the exponentials are recomputed in pass 3
//  instead of written back (the results are the same, bit for bit).
//  kPublish: the row list and its length are read by other blocks of the
//  launch, so they are written with device-scope stores.
template <int G, bool kShared, bool kPublish = false, int NT = kSelThreads>
__device__ __forceinline__ void select_after_max(double* __restrict__ lg, const double* s_m, int n_units, int n_pad,
                                                 int64_t s, int64_t ps, int units_cap, int budget,
                                                 const int32_t* __restrict__ unit_start,
                                                 int32_t* __restrict__ sel_units, int32_t* __restrict__ n_sel_units,
                                                 int32_t* __restrict__ n_sel, int32_t* __restrict__ row_ws,
                                                 double* __restrict__ scores_out, uint64_t* s_key, int* s_size,
                                                 int* s_incl) {
  constexpr int NW = NT / 64;
  static_assert(kSumThreads % NT == 0 && NT >= 128, "block size");
  __shared__ double s_rz[G][kSumThreads / 64];
  __shared__ double s_z[G];
  __shared__ int s_rtok[NW];
  __shared__ long long s_tok;
  __shared__ int s_ntake;
  __shared__ int s_wsum[NW];
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);

  // pass 2: exponentials and their sums per head.  The sums are taken as
  // kSumThreads threads would take them, whatever the block size: virtual
  // thread v sums the units v, v + kSumThreads, .. in increasing order, then
  // each virtual wave is summed over its lanes and the virtual waves in
  // order; a thread runs the virtual threads tid + k * NT (k < NV), so the
  // scores are the same bit for bit for every block size.  Up to kRegUnits
  // units per thread the logits are loaded in one batch and their
  // exponentials stay in registers for pass 3; beyond that they are kept in
  // the logit workspace (recomputed in pass 3 when other blocks wrote them).
  // The units' token count is summed on the way (it decides below which
  // search runs first).
  constexpr int kRegUnits = 4;
  constexpr int NV = kSumThreads / NT;   // virtual threads per thread
  constexpr int RV = kRegUnits / NV;     // register units per virtual thread
  static_assert(RV * NV == kRegUnits, "register units");
  const bool in_regs = n_units <= RV * kSumThreads;
  double ev[kRegUnits][G];
  double zs[NV][G];
  int tok = 0;
#pragma unroll
  for (int k = 0; k < NV; ++k)
#pragma unroll
    for (int j = 0; j < G; ++j) zs[k][j] = 0.0;
  if (in_regs) {
#pragma unroll
    for (int r = 0; r < kRegUnits; ++r) {
      const int u = tid + (r / RV) * NT + (r % RV) * kSumThreads;
#pragma unroll
      for (int j = 0; j < G; ++j) ev[r][j] = u < n_units ? load_logit<kShared>(lg + (size_t)u * G + j) : 0.0;
    }
#pragma unroll
    for (int r = 0; r < kRegUnits; ++r) {
      const int u = tid + (r / RV) * NT + (r % RV) * kSumThreads;
      if (u < n_units) {
        tok += s_size[u];
#pragma unroll
        for (int j = 0; j < G; ++j) {
          ev[r][j] = exp(ev[r][j] - s_m[j]);
          zs[r / RV][j] += ev[r][j];
        }
      }
    }
  } else {
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      for (int u = tid + k * NT; u < n_units; u += kSumThreads) {
        tok += s_size[u];
#pragma unroll
        for (int j = 0; j < G; ++j) {
          const double e = exp(load_logit<kShared>(lg + (size_t)u * G + j) - s_m[j]);
          if (!kShared) lg[(size_t)u * G + j] = e;
          zs[k][j] += e;
        }
      }
    }
  }
#pragma unroll
  for (int k = 0; k < NV; ++k)
#pragma unroll
    for (int j = 0; j < G; ++j) {
      const double z = wave_sum(zs[k][j]);
      if (lane == 0) s_rz[j][w + k * NW] = z;
    }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) tok += __shfl_xor(tok, o, kWave);
  if (lane == 0) s_rtok[w] = tok;
  __syncthreads();
  if (tid < G) {
    double z = 0.0;
    for (int q2 = 0; q2 < kSumThreads / 64; ++q2) z += s_rz[tid][q2];
    s_z[tid] = z;
  }
  if (tid == kWave) {
    long long t = 0;
    for (int q2 = 0; q2 < NW; ++q2) t += s_rtok[q2];
    s_tok = t;
  }
  __syncthreads();

  // pass 3: averaged probabilities and sort keys (padding keys 0 rank last)
  if (in_regs) {
#pragma unroll
    for (int r = 0; r < kRegUnits; ++r) {
      const int u = tid + (r / RV) * NT + (r % RV) * kSumThreads;
      if (u < n_pad) {
        uint64_t key = 0;
        if (u < n_units) {
          double a = 0.0;
#pragma unroll
          for (int j = 0; j < G; ++j) a += ev[r][j] / s_z[j];
          a /= (double)G;
          key = unit_key(a, u);
          if (scores_out) scores_out[(size_t)s * units_cap + u] = a;
        }
        s_key[u] = key;
      }
    }
  } else {
    for (int u = tid; u < n_pad; u += NT) {
      uint64_t key = 0;
      if (u < n_units) {
        double a = 0.0;
#pragma unroll
        for (int j = 0; j < G; ++j)
          a += (kShared ? exp(load_logit<kShared>(lg + (size_t)u * G + j) - s_m[j]) : lg[(size_t)u * G + j]) / s_z[j];
        a /= (double)G;
        key = unit_key(a, u);
        if (scores_out) scores_out[(size_t)s * units_cap + u] = a;
      }
      s_key[u] = key;
    }
  }
  __syncthreads();

  // The prefix stop (Section 3.1 budget; units taken in rank order until the
  // next one does not fit), first over the 128 highest keys: each wave sorts
  // its 128-key chunks of s_key in registers and keeps the 128 largest keys
  // it has seen (merge_top128), wave 0 merges the waves' lists, takes their
  // inclusive size sums and finds where the budget stops the prefix.  If it
  // stops inside those 128, or every unit fits, that is the selection (the
  // same units in the same order as the full search below); otherwise the
  // search below runs.  Tried when the budget holds fewer than kTopTry units
  // of the mean size, so that it rarely needs the full search after it.
  constexpr int kTopTry = 96;
  const int32_t* ustart = unit_start + (size_t)ps * units_cap;
  int32_t* rows = row_ws + (size_t)s * budget;
  __shared__ uint64_t s_top[NW][2 * kWave];
  __shared__ int s_fast;
  if (tid == 0) s_fast = 0;
  if ((long long)budget * n_units < (long long)kTopTry * s_tok) {
    {
      uint64_t t0 = 0, t1 = 0;
      bool have = false;
      for (int ch = w; ch * 2 * kWave < n_pad; ch += NW) {
        const int b = ch * 2 * kWave;
        uint64_t v0 = b + lane < n_pad ? s_key[b + lane] : 0;
        uint64_t v1 = b + kWave + lane < n_pad ? s_key[b + kWave + lane] : 0;
        sort128_desc(v0, v1, lane);
        if (have) {
          merge_top128(t0, t1, v0, v1, lane);
        } else {
          t0 = v0;
          t1 = v1;
          have = true;
        }
      }
      s_top[w][lane] = t0;
      s_top[w][kWave + lane] = t1;
    }
    __syncthreads();
    if (w == 0) {
      uint64_t t0 = s_top[0][lane], t1 = s_top[0][kWave + lane];
      for (int q2 = 1; q2 < NW; ++q2) merge_top128(t0, t1, s_top[q2][lane], s_top[q2][kWave + lane], lane);
      const int n_real = min(2 * kWave, n_units);   // the list's real keys (the rest are padding zeros)
      const int i0 = lane, i1 = kWave + lane;
      const int z0 = i0 < n_real ? s_size[key_unit(t0)] : 0;
      const int z1 = i1 < n_real ? s_size[key_unit(t1)] : 0;
      int x0 = z0, x1 = z1;
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const int y0 = __shfl_up(x0, o, kWave), y1 = __shfl_up(x1, o, kWave);
        if (lane >= o) {
          x0 += y0;
          x1 += y1;
        }
      }
      const long long inc0 = x0, inc1 = (long long)__shfl(x0, kWave - 1, kWave) + x1;
      const int ntake = __popcll(__builtin_amdgcn_ballot_w64(i0 < n_real && inc0 <= budget)) +
                        __popcll(__builtin_amdgcn_ballot_w64(i1 < n_real && inc1 <= budget));
      // the first unit left out must be a real key (nonzero), or every unit taken
      const int nb = ntake < kWave ? ntake : ntake - kWave;
      const uint64_t k0 = ((uint64_t)(uint32_t)__shfl((int)(uint32_t)(t0 >> 32), nb & (kWave - 1), kWave) << 32) |
                          (uint32_t)__shfl((int)(uint32_t)t0, nb & (kWave - 1), kWave);
      const uint64_t k1 = ((uint64_t)(uint32_t)__shfl((int)(uint32_t)(t1 >> 32), nb & (kWave - 1), kWave) << 32) |
                          (uint32_t)__shfl((int)(uint32_t)t1, nb & (kWave - 1), kWave);
      const uint64_t kb = ntake < kWave ? k0 : k1;
      const bool fast = ntake < n_real ? kb != 0 : n_real == n_units;
      if (fast) {
        if (i0 < ntake) {
          const int u = key_unit(t0);
          sel_units[(size_t)s * units_cap + i0] = u;
          s_key[i0] = ((uint64_t)(uint32_t)ustart[u] << 32) | (uint32_t)z0;
          s_incl[i0] = inc0 > 0x3fffffff ? 0x3fffffff : (int)inc0;
        }
        if (i1 < ntake) {
          const int u = key_unit(t1);
          sel_units[(size_t)s * units_cap + i1] = u;
          s_key[i1] = ((uint64_t)(uint32_t)ustart[u] << 32) | (uint32_t)z1;
          s_incl[i1] = inc1 > 0x3fffffff ? 0x3fffffff : (int)inc1;
        }
      }
      if (lane == 0) {
        s_fast = fast ? 1 : 0;
        if (fast) s_ntake = ntake;
      }
    }
  }
  __syncthreads();
  if (!s_fast) {
    // The full search: radix selection.  The boundary unit is the first
    // one in rank order whose size exceeds what the units ranked above it leave
    // of the budget.  Keys are distinct, so 8-bit digits from the top narrow
    // the candidates to the bucket in which the token count of the higher keys
    // crosses the remaining budget, until that bucket holds one unit; every
    // unit with a higher key is taken.  Then only the taken units are sorted.
    // Histograms per pair of waves: a unit adds (size << 16) + 1 to its digit's
    // entry, so one 64-bit word counts tokens (bits 16..) and units (bits
    // 0..15; at most kMaxUnits per slice), and LDS atomics conflict only inside
    // a pair.  Two sets alternate between passes, so a pass clears the other
    // set while its own is scanned (2 x 4 x 256 words: 16 KiB of LDS).
    // Leading bytes that every key shares (the sign and high exponent bits of
    // the scores) are skipped: the search starts at the first byte where the
    // keys' OR and AND differ.
    constexpr int kHists = NW / 2;
    __shared__ uint64_t s_hist[2][kHists][256];
    __shared__ uint64_t s_or[NW], s_and[NW];
    __shared__ uint64_t s_prefix, s_thresh;
    __shared__ int64_t s_rem;
    __shared__ int s_pbits, s_state, s_nsel_units;   // state: 0 searching, 1 boundary found, 2 every unit fits
    {
      uint64_t ko = 0, ka = ~0ull;
      for (int u = tid; u < n_units; u += NT) {
        ko |= s_key[u];
        ka &= s_key[u];
      }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        ko |= __shfl_xor(ko, o, kWave);
        ka &= __shfl_xor(ka, o, kWave);
      }
      if (lane == 0) {
        s_or[w] = ko;
        s_and[w] = ka;
      }
    }
    for (int i = tid; i < 2 * kHists * 256; i += NT) (&s_hist[0][0][0])[i] = 0;
    __syncthreads();
    if (tid == 0) {
      uint64_t ko = 0, ka = ~0ull;
      for (int q2 = 0; q2 < NW; ++q2) {
        ko |= s_or[q2];
        ka &= s_and[q2];
      }
      const uint64_t diff = ko ^ ka;          // bits where the keys differ
      const int lead = diff ? __builtin_clzll(diff) / 8 * 8 : 56;   // whole shared bytes
      s_pbits = lead;
      s_prefix = lead ? (ko >> (64 - lead)) : 0;
      s_rem = budget;
      s_state = 0;
      s_nsel_units = 0;
    }
    __syncthreads();
    int set = 0;
    while (s_state == 0) {
      const int pbits = s_pbits;
      const uint64_t prefix = s_prefix;
      const int shift = 56 - pbits;
      for (int u = tid; u < n_units; u += NT) {
        const uint64_t k = s_key[u];
        if (pbits == 0 || (k >> (64 - pbits)) == prefix) {
          const int dg = (int)((k >> shift) & 255u);
          atomicAdd(reinterpret_cast<unsigned long long*>(&s_hist[set][w % kHists][dg]),
                    ((unsigned long long)(uint32_t)s_size[key_unit(k)] << 16) + 1ull);
        }
      }
      __syncthreads();
      if (w == 0) {
        // lane l holds digits 255 - 4l .. 252 - 4l, highest first
        // (a slice's tokens, hence every sum below, stay under 2^31)
        int v[4];
        int cnt[4];
        int tot = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          uint64_t h = 0;
#pragma unroll
          for (int q2 = 0; q2 < kHists; ++q2) h += s_hist[set][q2][255 - 4 * lane - i];
          v[i] = (int)(h >> 16);
          cnt[i] = (int)(h & 0xffffu);
          tot += v[i];
        }
        int incl = tot;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int y = __shfl_up(incl, o, kWave);
          if (lane >= o) incl += y;
        }
        int64_t cum = incl - tot;   // tokens of the digits above this lane's
        const int64_t rem = s_rem;
        int hit = -1, hit_cnt = 0;
        int64_t before = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (hit < 0 && cum + v[i] > rem) {
            hit = 255 - 4 * lane - i;
            hit_cnt = cnt[i];
            before = cum;
          }
          cum += v[i];
        }
        const uint64_t found = __builtin_amdgcn_ballot_w64(hit >= 0);
        if (found == 0) {
          if (lane == 0) s_state = 2;    // the candidates are every unit (first pass) and all fit
        } else if (lane == (int)__builtin_ctzll(found)) {
          s_prefix = (prefix << 8) | (uint64_t)hit;
          s_rem = rem - before;
          s_pbits = pbits + 8;
          if (hit_cnt == 1 || pbits + 8 == 64) s_state = 1;
        }
      } else {
        for (int i = tid - 64; i < kHists * 256; i += NT - 64) (&s_hist[set ^ 1][0][0])[i] = 0;
      }
      set ^= 1;
      __syncthreads();
    }
    if (s_state == 1) {
      // the boundary unit is the one key under the final prefix
      const int pb = s_pbits;
      const uint64_t pf = s_prefix;
      for (int u = tid; u < n_units; u += NT) {
        const uint64_t k = s_key[u];
        if ((pb == 64 ? k : (k >> (64 - pb))) == pf) s_thresh = k;
      }
    }
    __syncthreads();
    // the taken keys, compacted to the front of s_key and sorted there
    const bool take_all = s_state == 2;
    const uint64_t thresh = take_all ? 0 : s_thresh;
    constexpr int kPerThread = kMaxUnits / NT;
    uint64_t mine[kPerThread];
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const int u = tid + i * NT;
      mine[i] = u < n_units ? s_key[u] : 0;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const int u = tid + i * NT;
      if (u < n_units && (take_all || mine[i] > thresh)) s_key[atomicAdd(&s_nsel_units, 1)] = mine[i];
    }
    __syncthreads();
    const int n_taken = s_nsel_units;
    n_pad = 64;
    while (n_pad < n_taken) n_pad <<= 1;
    for (int i = n_taken + tid; i < n_pad; i += NT) s_key[i] = 0;   // padding ranks last
    __syncthreads();

    // bitonic sort, descending keys (n_pad >= 64)
    // (chunks c and c + NW of a wave go together; a missing second
    // chunk is a copy of the first, sorted and dropped)
    const int n_chunk = n_pad / 64;
    for (int c = w; c < n_chunk; c += 2 * NW) {
      const int c1 = c + NW < n_chunk ? c + NW : c;
      const int i0 = 64 * c + lane, i1 = 64 * c1 + lane;
      uint64_t v0 = s_key[i0], v1 = s_key[i1];
#pragma unroll
      for (int k = 2; k <= 64; k <<= 1) bitonic_in_wave2(v0, v1, i0, i1, k, k >> 1);
      s_key[i0] = v0;
      if (c1 != c) s_key[i1] = v1;
    }
    __syncthreads();
    for (int k = 128; k <= n_pad; k <<= 1) {
      for (int jj = k >> 1; jj >= 64; jj >>= 1) {
        // pair t: i has a zero at bit jj, its partner p = i + jj
        for (int t = tid; t < n_pad / 2; t += NT) {
          const int i = ((t & ~(jj - 1)) << 1) | (t & (jj - 1));
          const int p = i | jj;
          const uint64_t a = s_key[i], b = s_key[p];
          const bool desc = (i & k) == 0;
          if (desc ? a < b : a > b) {
            s_key[i] = b;
            s_key[p] = a;
          }
        }
        __syncthreads();
      }
      for (int c = w; c < n_chunk; c += 2 * NW) {
        const int c1 = c + NW < n_chunk ? c + NW : c;
        const int i0 = 64 * c + lane, i1 = 64 * c1 + lane;
        uint64_t v0 = s_key[i0], v1 = s_key[i1];
        bitonic_in_wave2(v0, v1, i0, i1, k, 32);
        s_key[i0] = v0;
        if (c1 != c) s_key[i1] = v1;
      }
      __syncthreads();
    }

    // inclusive size sums in rank order (all within the budget by construction)
    if (tid == 0) s_ntake = 0;
    int carry = 0;
    for (int base = 0; base < n_taken; base += NT) {
      const int p = base + tid;
      const int v = p < n_taken ? s_size[key_unit(s_key[p])] : 0;
      int x = v;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
      }
      if (lane == 63) s_wsum[w] = x;
      __syncthreads();
      int wp = 0;
      for (int q2 = 0; q2 < w; ++q2) wp += s_wsum[q2];
      const long long inc = (long long)carry + wp + x;
      if (p < n_taken) {
        s_incl[p] = inc > 0x3fffffff ? 0x3fffffff : (int)inc;   // sums past the budget are never read
        if (inc <= budget) atomicAdd(&s_ntake, 1);
      }
      int tot = 0;
      for (int q2 = 0; q2 < NW; ++q2) tot += s_wsum[q2];
      carry = (int)std::min<long long>((long long)carry + tot, 0x3fffffff);
      __syncthreads();
    }
    // the unit list in rank order; each rank's key slot then holds its unit's
    // first pool row and size (the starts loaded together, one per thread)
    const int ntake_full = s_ntake;
    for (int p = tid; p < ntake_full; p += NT) {
      const int u = key_unit(s_key[p]);
      sel_units[(size_t)s * units_cap + p] = u;
      s_key[p] = ((uint64_t)(uint32_t)ustart[u] << 32) | (uint32_t)s_size[u];
    }
  }
  __syncthreads();
  const int ntake = s_ntake;
  const int nsel = ntake > 0 ? s_incl[ntake - 1] : 0;
  // one wave per selected unit: its rows in order
  for (int p = w; p < ntake; p += NW) {
    const uint64_t e = s_key[p];
    const int sz = (int)(uint32_t)e;
    const int st0 = (int)(uint32_t)(e >> 32);
    const int ex = s_incl[p] - sz;
    for (int i = lane; i < sz; i += kWave) {
      if constexpr (kPublish)
        __hip_atomic_store(rows + ex + i, st0 + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      else
        rows[ex + i] = st0 + i;
    }
  }
  if (tid == 0) {
    n_sel_units[s] = ntake;
    if constexpr (kPublish)
      __hip_atomic_store(n_sel + s, nsel, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
      n_sel[s] = nsel;
  }
}

// One block per fired slice: the float64 group-consistent scores (Appendix B),
// a descending bitonic sort of the unit keys, prefix-stop under the budget,
// the selected unit list and the pool-row list that the gather kernel copies.
//  pass 1  the logits and their maxima M_j: with own_logits the block computes
//          them as unit_logits_kernel does (one block per slice fills the
//          chip when many slices fire); otherwise unit_logits_kernel has
//          written them, spread over several blocks per slice.  The unit
//          sizes go to LDS.
//  pass 2  e_ju = exp(l_ju - M_j) and Z_j = sum_u e_ju.
//  pass 3  A_u = (1/g) sum_j e_ju / Z_j and the sort keys.
//  sort    64-key chunks in registers for merge distances below 64 (no
//          barrier), LDS steps with a barrier for the longer ones.
template <class T, int G, int NT>
__global__ __launch_bounds__(NT)
void score_select_kernel(const T* __restrict__ q, int n_kv_heads, double scale, const float* __restrict__ reps,
                         const int32_t* __restrict__ unit_start, const int32_t* __restrict__ unit_size,
                         int units_cap, int n_units_arg, int budget, const uint8_t* __restrict__ fire,
                         int32_t* __restrict__ sel_units, int32_t* __restrict__ n_sel_units,
                         int32_t* __restrict__ n_sel, double* __restrict__ scores_out,
                         double* __restrict__ logit_ws, int32_t* __restrict__ row_ws, int n_pad_arg,
                         const int32_t* __restrict__ seg_state, int seg_stride, int slice_div, int own_logits) {
  extern __shared__ __align__(16) char smem[];
  uint64_t* s_key = reinterpret_cast<uint64_t*>(smem);            // [n_pad_arg]
  int* s_size = reinterpret_cast<int*>(s_key + n_pad_arg);        // [n_pad_arg] unit sizes by unit id
  int* s_incl = s_size + n_pad_arg;                                // [n_pad_arg] inclusive size sums by rank
  constexpr int NW = NT / 64;
  __shared__ double s_rm[G][NW];
  __shared__ double s_m[G];

  const int64_t s = blockIdx.x;
  const int64_t grp = s / n_kv_heads;
  if (fire && !fire[grp]) return;
  // slice_div > 1: per-head selection, s is a query head and ps the slice of
  // its KV head, whose units it ranks alone
  const int64_t ps = s / slice_div;
  // with boundary-delimited segments each slice has its own unit count (the
  // argument is then an upper bound that sized the LDS)
  const int n_units = slice_units(seg_state, seg_stride, ps, n_units_arg);
  int n_pad = n_pad_arg;
  if (seg_state) {
    n_pad = 64;
    while (n_pad < n_units) n_pad <<= 1;
  }
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int32_t* us = unit_size + (size_t)ps * units_cap;
  for (int u = tid; u < n_units; u += NT) s_size[u] = max(us[u], 0);

  // pass 1: maxima of the logits, computed here (own_logits: many slices,
  // one block each) or read back from unit_logits_kernel (few slices)
  double mx[G];
#pragma unroll
  for (int j = 0; j < G; ++j) mx[j] = -__builtin_inf();
  double* lg = logit_ws + (size_t)s * units_cap * G;
  if (own_logits) {
    const int kvh = (int)(s - grp * n_kv_heads);
    const int n_q_heads = n_kv_heads * G;
    double qd[G][LogitLayout<G>::kDims];
    load_q_f64<G>(q, (size_t)grp * n_q_heads + (size_t)kvh * G, lane, qd);
    const float* rs = reps + (size_t)ps * units_cap * kHeadDim;
    for (int u0 = w * kLogitUnitsPerIter; u0 < n_units; u0 += NW * kLogitUnitsPerIter)
      wave_unit_logits<G, false>(qd, rs, u0, n_units, scale, lg, mx, lane);
  } else {
    for (int u = tid; u < n_units; u += NT) {
#pragma unroll
      for (int j = 0; j < G; ++j) mx[j] = fmax(mx[j], lg[(size_t)u * G + j]);
    }
  }
#pragma unroll
  for (int j = 0; j < G; ++j) {
    const double m = wave_max(mx[j]);
    if (lane == 0) s_rm[j][w] = m;
  }
  __syncthreads();
  if (tid < G) {
    double m = s_rm[tid][0];
    for (int q2 = 1; q2 < NW; ++q2) m = fmax(m, s_rm[tid][q2]);
    s_m[tid] = m;
  }
  __syncthreads();

  select_after_max<G, false, false, NT>(lg, s_m, n_units, n_pad, s, ps, units_cap, budget, unit_start, sel_units, n_sel_units,
                             n_sel, row_ws, scores_out, s_key, s_size, s_incl);
}

// A fired slice's part `part` of the selection work in a decode step: the
// logits of the part's units and their per-head maxima, written with
// device-scope stores; the part then counts itself in at the slice's
// counter (`counter`), and the last part to arrive resets it, loads every part's maxima
// and the unit sizes and makes the selection (select_after_max, the same
// code as the per-stage kernel, so scores and selections are equal bit for
// bit).  Returns true in the block that made the selection.
template <class T, int G, bool kPublish>
__device__ __forceinline__ bool select_part(const T* __restrict__ q, int n_kv_heads, int64_t s, int part, int n_parts,
                                            double scale, const float* __restrict__ reps, int units_cap, int n_units,
                                            int n_pad, int budget, const int32_t* __restrict__ unit_start,
                                            const int32_t* __restrict__ unit_size, int32_t* __restrict__ sel_units,
                                            int32_t* __restrict__ n_sel_units, int32_t* __restrict__ n_sel,
                                            int32_t* __restrict__ sel_rows, double* __restrict__ scores_out,
                                            double* __restrict__ logit_ws, double* __restrict__ part_max,
                                            int32_t* __restrict__ counter, char* smem) {
  uint64_t* s_key = reinterpret_cast<uint64_t*>(smem);            // [n_pad]
  int* s_size = reinterpret_cast<int*>(s_key + n_pad);            // [n_pad] unit sizes by unit id
  int* s_incl = s_size + n_pad;                                    // [n_pad] inclusive size sums by rank
  __shared__ double s_rm[G][kSelWaves];
  __shared__ double s_m[G];
  __shared__ int s_last;
  const int64_t grp = s / n_kv_heads;
  const int kvh = (int)(s - grp * n_kv_heads);
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n_q_heads = n_kv_heads * G;

  // logits of this part's units and their maxima
  const int per = (n_units + n_parts - 1) / n_parts;
  const int u_begin = part * per, u_end = min(n_units, u_begin + per);
  double mx[G];
#pragma unroll
  for (int j = 0; j < G; ++j) mx[j] = -__builtin_inf();
  double* lg = logit_ws + (size_t)s * units_cap * G;
  if (u_begin < u_end) {
    double qd[G][LogitLayout<G>::kDims];
    load_q_f64<G>(q, (size_t)grp * n_q_heads + (size_t)kvh * G, lane, qd);
    const float* rs = reps + (size_t)s * units_cap * kHeadDim;
    for (int u0 = u_begin + w * kLogitUnitsPerIter; u0 < u_end; u0 += kSelWaves * kLogitUnitsPerIter)
      wave_unit_logits<G, true>(qd, rs, u0, u_end, scale, lg, mx, lane);
  }
#pragma unroll
  for (int j = 0; j < G; ++j) {
    const double m = wave_max(mx[j]);
    if (lane == 0) s_rm[j][w] = m;
  }
  __syncthreads();
  if (tid < G) {
    double m = s_rm[tid][0];
    for (int q2 = 1; q2 < kSelWaves; ++q2) m = fmax(m, s_rm[tid][q2]);
    __hip_atomic_store(part_max + ((size_t)s * n_parts + part) * G + tid, m, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  }
  // count this part in once its stores are done; the last one selects
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (tid == 0) {
    const int old = __hip_atomic_fetch_add(counter, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_last = old == n_parts - 1;
    if (s_last) __hip_atomic_store(counter, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (!s_last) return false;
  // the parts' maxima (one coherent load per thread, all in flight) and the unit sizes
  __shared__ double s_pmax[kMaxSelectParts * kMaxGroupSize];
  if (tid < n_parts * G)
    s_pmax[tid] = __hip_atomic_load(part_max + (size_t)s * n_parts * G + tid, __ATOMIC_RELAXED,
                                    __HIP_MEMORY_SCOPE_AGENT);
  const int32_t* us = unit_size + (size_t)s * units_cap;
  for (int u = tid; u < n_units; u += kSelThreads) s_size[u] = max(us[u], 0);
  __syncthreads();
  if (tid < G) {
    double m = -__builtin_inf();
    for (int p2 = 0; p2 < n_parts; ++p2) m = fmax(m, s_pmax[p2 * G + tid]);
    s_m[tid] = m;
  }
  __syncthreads();
  select_after_max<G, true, kPublish>(lg, s_m, n_units, n_pad, s, s, units_cap, budget, unit_start, sel_units,
                                      n_sel_units, n_sel, sel_rows, scores_out, s_key, s_size, s_incl);
  return true;
}

// The first launch of a two-launch decode step (fixed segments): one
// 512-thread block per (slice, part of its units).  Every block computes its
// group's r (the same float64 value in every block; one block per group
// writes it and the decision), block 0 of a slice runs the fixed-segment
// store (window append and oldest-segment eviction on its first wave: it
// writes only the unit it creates and rows past every existing unit, which
// the retrieval does not read), and if the group fired each block does its
// part of the selection (select_part).  The reference query is left for the
// attention launch to update.
template <class T, int G>
__global__ __launch_bounds__(kSelThreads)
void step_select_kernel(const T* __restrict__ q, const T* __restrict__ q_ref, int n_kv_heads, double tau, int first,
                        double* __restrict__ r_out, uint8_t* __restrict__ fire_out, const T* __restrict__ k_new,
                        const T* __restrict__ v_new, T* __restrict__ k_local, T* __restrict__ v_local, int window,
                        int step, int seg_len, int evict_seg, float* __restrict__ reps,
                        int32_t* __restrict__ unit_start, int32_t* __restrict__ unit_size, int units_cap,
                        int n_clusters, T* __restrict__ k_pool, T* __restrict__ v_pool, int64_t pool_rows,
                        int prompt_len, double scale, int n_units, int budget, int32_t* __restrict__ sel_units,
                        int32_t* __restrict__ n_sel_units, int32_t* __restrict__ n_sel,
                        int32_t* __restrict__ sel_rows, double* __restrict__ scores_out,
                        double* __restrict__ logit_ws, double* __restrict__ part_max, int32_t* __restrict__ counter,
                        int n_parts, int n_pad) {
  extern __shared__ __align__(16) char smem[];
  __shared__ double s_bpart[16];
  const int64_t s = blockIdx.x / n_parts;
  const int part = (int)(blockIdx.x - s * n_parts);
  const int64_t grp = s / n_kv_heads;
  const int kvh = (int)(s - grp * n_kv_heads);
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);

  const double r = boundary_r(q, q_ref, n_kv_heads * G, first, grp, s_bpart);
  const bool fire = first || r < tau;
  if (part == 0 && kvh == 0 && tid == 0) {
    if (r_out) r_out[grp] = r;
    fire_out[grp] = (uint8_t)(fire ? 1 : 0);
  }
  if (part == 0 && w == 0)
    store_slice(k_new, v_new, k_local, v_local, window, step, seg_len, evict_seg, reps, unit_start, unit_size,
                units_cap, n_clusters, k_pool, v_pool, pool_rows, prompt_len, s, lane);
  if (!fire) return;
  select_part<T, G, false>(q, n_kv_heads, s, part, n_parts, scale, reps, units_cap, n_units, n_pad, budget,
                           unit_start, unit_size, sel_units, n_sel_units, n_sel, sel_rows, scores_out, logit_ws,
                           part_max, counter + s, smem);
}

// Copy selected pool rows into KV_critical: 16 lanes per row, 16 rows per pass.
template <class T>
__global__ __launch_bounds__(256)
void gather_kernel(const T* __restrict__ k_pool, const T* __restrict__ v_pool, int64_t pool_rows,
                   const int32_t* __restrict__ row_ws, const int32_t* __restrict__ n_sel,
                   const uint8_t* __restrict__ fire, int n_kv_heads, int budget, int blocks_per_slice,
                   int rows_per_block, T* __restrict__ k_buf, T* __restrict__ v_buf) {
  const int64_t s = blockIdx.x / blocks_per_slice;
  const int b = (int)(blockIdx.x - s * blocks_per_slice);
  if (fire && !fire[s / n_kv_heads]) return;
  const int n = n_sel[s];
  const int r0 = b * rows_per_block;
  if (r0 >= n) return;
  const int r1 = min(n, r0 + rows_per_block);
  constexpr int kU4 = kHeadDim * sizeof(T) / 16;     // 16 (bf16) or 32 (fp32)
  const int sub = threadIdx.x & 15;
  const int32_t* rows = row_ws + (size_t)s * budget;
  for (int r = r0 + (threadIdx.x >> 4); r < r1; r += 16) {
    const int64_t pr = rows[r];
    if (pr < 0 || pr >= pool_rows) continue;   // unit table pointing outside the pool
    const uint4* ks = reinterpret_cast<const uint4*>(k_pool + ((size_t)s * pool_rows + pr) * kHeadDim);
    const uint4* vs = reinterpret_cast<const uint4*>(v_pool + ((size_t)s * pool_rows + pr) * kHeadDim);
    uint4* kd = reinterpret_cast<uint4*>(k_buf + ((size_t)s * budget + r) * kHeadDim);
    uint4* vd = reinterpret_cast<uint4*>(v_buf + ((size_t)s * budget + r) * kHeadDim);
#pragma unroll
    for (int q = sub; q < kU4; q += 16) {
      const uint4 a = ks[q], c = vs[q];
      kd[q] = a;
      vd[q] = c;
    }
  }
}

// ------------------------------------------------------------------ delta gather
//
// KV_critical as a cache of pool rows (the delta transfer of a host-resident
// pool).  buf_row[s][i] is the pool row held in buffer slot i (-1: free).  For
// a fired slice the plan kernel keeps every slot whose row is selected again,
// frees the others, and pairs the newly selected rows (selection order) with
// the free slots (slot order); only those rows cross the host link (fetch
// kernel).  slot_list then lists the n_sel slots holding the selection, which
// the row-list attention reads from the buffers.

constexpr int kPlanThreads = 1024;
constexpr int64_t kDeltaMaxPoolRows = 512 * 1024;   // the plan's bitmap of pool rows fits 64 KiB of LDS
constexpr int kPlanWaves = kPlanThreads / 64;

// Exclusive block-wide prefix sum of one flag per thread; returns the total.
__device__ __forceinline__ int block_scan_flag(int flag, int* s_w, int& excl) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const uint64_t m = __builtin_amdgcn_ballot_w64(flag != 0);
  const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
  if (lane == 0) s_w[w] = __popcll(m);
  __syncthreads();
  int before = 0, total = 0;
  for (int q = 0; q < kPlanWaves; ++q) {
    const int c = s_w[q];
    before += q < w ? c : 0;
    total += c;
  }
  __syncthreads();
  excl = before + below;
  return total;
}

// Exclusive block-wide prefix sum of one count per thread; returns the total.
__device__ __forceinline__ int block_scan_count(int c, int* s_w, int& excl) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int incl = c;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o, kWave);
    if (lane >= o) incl += y;
  }
  if (lane == 63) s_w[w] = incl;
  __syncthreads();
  int before = 0, total = 0;
  for (int q = 0; q < kPlanWaves; ++q) {
    const int x = s_w[q];
    before += q < w ? x : 0;
    total += x;
  }
  __syncthreads();
  excl = before + incl - c;
  return total;
}

__global__ __launch_bounds__(kPlanThreads)
void delta_plan_kernel(const int32_t* __restrict__ row_ws, const int32_t* __restrict__ n_sel,
                       const uint8_t* __restrict__ fire, int n_kv_heads, int budget, int64_t pool_rows,
                       int32_t* __restrict__ buf_row, int32_t* __restrict__ slot_list,
                       int32_t* __restrict__ fetch_slot, int32_t* __restrict__ fetch_row,
                       int32_t* __restrict__ n_fetch, int32_t* __restrict__ n_fetch_out) {
  extern __shared__ uint32_t s_bits[];   // one bit per pool row
  __shared__ int s_w[kPlanWaves];
  __shared__ int s_base[3];
  const int64_t s = blockIdx.x;
  const int tid = threadIdx.x;
  if (fire && !fire[s / n_kv_heads]) {
    if (tid == 0) {
      n_fetch[s] = 0;
      if (n_fetch_out) n_fetch_out[s] = 0;
    }
    return;
  }
  const int n = min(max(n_sel[s], 0), budget);
  const int words = (int)((pool_rows + 31) / 32);
  const int32_t* rows = row_ws + (size_t)s * budget;
  int32_t* brow = buf_row + (size_t)s * budget;
  for (int i = tid; i < words; i += kPlanThreads) s_bits[i] = 0u;
  __syncthreads();
  for (int p = tid; p < n; p += kPlanThreads) {
    const int r = rows[p];
    if (r >= 0 && r < pool_rows) atomicOr(&s_bits[r >> 5], 1u << (r & 31));
  }
  __syncthreads();
  // keep the slots whose row is selected again (test and clear its bit), free the rest
  for (int i = tid; i < budget; i += kPlanThreads) {
    const int r = brow[i];
    bool keep = false;
    if (r >= 0 && r < pool_rows) {
      const uint32_t bit = 1u << (r & 31);
      keep = (atomicAnd(&s_bits[r >> 5], ~bit) & bit) != 0;
    }
    if (!keep) brow[i] = -1;
  }
  __syncthreads();
  // pair the k-th new row (selection order) with the k-th free slot (slot order)
  if (tid == 0) { s_base[0] = 0; s_base[1] = 0; }
  __syncthreads();
  const int rounds = (budget + kPlanThreads - 1) / kPlanThreads;
  for (int rd = 0; rd < rounds; ++rd) {
    // free slots of this round
    const int i = rd * kPlanThreads + tid;
    const bool fr = i < budget && brow[i] < 0;
    int ex;
    const int tot = block_scan_flag(fr, s_w, ex);
    if (fr) fetch_slot[(size_t)s * budget + s_base[1] + ex] = i;
    __syncthreads();
    if (tid == 0) s_base[1] += tot;
    __syncthreads();
  }
  for (int rd = 0; rd < rounds; ++rd) {
    const int p = rd * kPlanThreads + tid;
    int r = -1;
    bool nw = false;
    if (p < n) {
      r = rows[p];
      nw = r >= 0 && r < pool_rows && (s_bits[r >> 5] >> (r & 31) & 1u);
    }
    int ex;
    const int tot = block_scan_flag(nw, s_w, ex);
    if (nw) {
      const int k = s_base[0] + ex;            // k < number of free slots (the selection fits the buffer)
      const int slot = fetch_slot[(size_t)s * budget + k];
      fetch_row[(size_t)s * budget + k] = r;
      brow[slot] = r;
    }
    __syncthreads();
    if (tid == 0) s_base[0] += tot;
    __syncthreads();
  }
  if (tid == 0) {
    n_fetch[s] = s_base[0];
    if (n_fetch_out) n_fetch_out[s] = s_base[0];
  }
  __syncthreads();
  // the slots that hold the selection, in slot order
  if (tid == 0) s_base[2] = 0;
  __syncthreads();
  for (int rd = 0; rd < rounds; ++rd) {
    const int i = rd * kPlanThreads + tid;
    const bool v = i < budget && brow[i] >= 0;
    int ex;
    const int tot = block_scan_flag(v, s_w, ex);
    if (v && s_base[2] + ex < budget) slot_list[(size_t)s * budget + s_base[2] + ex] = i;
    __syncthreads();
    if (tid == 0) s_base[2] += tot;
    __syncthreads();
  }
}

// KV_critical as an LRU cache of pool rows: cache_rows >= budget slots per
// slice, slot_step[s][i] the decode step at which slot i's row was last
// selected (-1: empty).  For a fired slice at decode step `step`:
//  - every slot whose row is selected again keeps it (slot_step = step);
//  - the k newly selected rows (selection order) go to the k other slots with
//    the smallest (slot_step, slot), paired in slot order: empty slots first,
//    then the rows selected longest ago;
//  - slot_list lists the n_sel slots holding the selection, in slot order.
// Thread t holds slots [R t, R t + R) in registers for the whole plan.  The
// k-th smallest key slot_step + 1 among the candidates (slots not selected
// now) comes from a radix select by 8-bit digits (per-wave histograms), the
// ties at the threshold in slot order from block scans.
constexpr int kCacheMaxStep = (1 << 24) - 2;
constexpr int kCacheMaxSlotsPerThread = 64;
constexpr int kCacheMaxRows = kPlanThreads * kCacheMaxSlotsPerThread;

// x[j] = a[i0 + j] for j < R (fill past n), in 16-byte loads where the run
// is aligned and whole (a thread's run is consecutive, so a wave's plain
// loads would each touch 64 lines)
template <int R>
__device__ __forceinline__ void load_run(const int32_t* a, int i0, int n, int fill, int (&x)[R]) {
  const bool vec = ((reinterpret_cast<uintptr_t>(a + i0) & 15u) == 0) && i0 + R <= n;
  if (vec) {
#pragma unroll
    for (int j = 0; j < R; j += 4) {
      const int4 v = *reinterpret_cast<const int4*>(a + i0 + j);
      x[j] = v.x;
      x[j + 1] = v.y;
      x[j + 2] = v.z;
      x[j + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int j = 0; j < R; ++j) x[j] = i0 + j < n ? a[i0 + j] : fill;
  }
}

template <int R>
__global__ __launch_bounds__(kPlanThreads)
void cache_plan_kernel(const int32_t* __restrict__ row_ws, const int32_t* __restrict__ n_sel,
                       const uint8_t* __restrict__ fire, int n_kv_heads, int budget, int cache_rows,
                       int64_t pool_rows, int step, int32_t* __restrict__ buf_row, int32_t* __restrict__ slot_step,
                       int32_t* __restrict__ slot_list, int32_t* __restrict__ fetch_slot,
                       int32_t* __restrict__ fetch_row, int32_t* __restrict__ n_fetch,
                       int32_t* __restrict__ n_fetch_out) {
  extern __shared__ uint32_t s_bits[];   // one bit per pool row
  __shared__ int s_w[kPlanWaves];
  __shared__ int s_hist[kPlanWaves][256];
  __shared__ int s_k, s_below, s_thr;
  const int64_t s = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (fire && !fire[s / n_kv_heads]) {
    if (tid == 0) {
      n_fetch[s] = 0;
      if (n_fetch_out) n_fetch_out[s] = 0;
    }
    return;
  }
  const int n = min(max(n_sel[s], 0), budget);
  const int words = (int)((pool_rows + 31) / 32);
  const int32_t* rows = row_ws + (size_t)s * budget;
  int32_t* brow = buf_row + (size_t)s * cache_rows;
  int32_t* bstep = slot_step + (size_t)s * cache_rows;
  const int i0 = tid * R;
  // key[j] = slot_step + 1 of slot i0 + j (0: empty); slots past the end
  // take step + 1, which is never a candidate
  int key[R];
  load_run<R>(bstep, i0, cache_rows, step, key);
#pragma unroll
  for (int j = 0; j < R; ++j) key[j] += 1;
  for (int i = tid; i < words; i += kPlanThreads) s_bits[i] = 0u;
  if (tid == 0) s_k = 0;
  __syncthreads();
  for (int p = tid; p < n; p += kPlanThreads) {
    const int r = rows[p];
    if (r >= 0 && r < pool_rows) atomicOr(&s_bits[r >> 5], 1u << (r & 31));
  }
  __syncthreads();
  // hits: slots whose row is selected again (test and clear its bit); the
  // thread's own run only, read in pieces of up to 16 slots
  constexpr int kPiece = R < 16 ? R : 16;
  static_assert(R % kPiece == 0, "a run splits into whole pieces");
  uint64_t hit = 0;
#pragma unroll
  for (int j0 = 0; j0 < R; j0 += kPiece) {
    int row[kPiece];
    load_run<kPiece>(brow, i0 + j0, cache_rows, -1, row);
#pragma unroll
    for (int j = 0; j < kPiece; ++j) {
      const int r = row[j];
      if (r >= 0 && r < pool_rows) {
        const uint32_t bit = 1u << (r & 31);
        if (atomicAnd(&s_bits[r >> 5], ~bit) & bit) hit |= 1ull << (j0 + j);
      }
    }
  }
#pragma unroll
  for (int j = 0; j < R; ++j)
    if (hit >> j & 1ull) {
      key[j] = step + 1;
      bstep[i0 + j] = step;
    }
  __syncthreads();
  // the new rows: still marked
  int kk = 0;
  for (int p = tid; p < n; p += kPlanThreads) {
    const int r = rows[p];
    kk += (r >= 0 && r < pool_rows && (s_bits[r >> 5] >> (r & 31) & 1u)) ? 1 : 0;
  }
  kk = wave_sum_int(kk);
  if (lane == 0) atomicAdd(&s_k, kk);
  __syncthreads();
  const int k = s_k;
  // radix select of the k-th smallest candidate key, from the highest digit
  // that step + 1 uses
  int below = 0;   // candidates with a key below the prefix's range, taken whole
  int prefix = 0;
  const int top = step < 255 ? 0 : step < 65535 ? 8 : 16;
  for (int shift = top; shift >= 0 && k > 0; shift -= 8) {
    for (int i = tid; i < kPlanWaves * 256; i += kPlanThreads) (&s_hist[0][0])[i] = 0;
    __syncthreads();
    // runs of one digit are counted in a register and added once; a thread's
    // last run is added once per wave when the wave's agree
    int cur = -1, cnt = 0;
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const int x = key[j];
      if (x <= step && (x >> (shift + 8)) == prefix) {
        const int dg = (x >> shift) & 255;
        if (dg != cur) {
          if (cnt) atomicAdd(&s_hist[wv][cur], cnt);
          cur = dg;
          cnt = 0;
        }
        ++cnt;
      }
    }
    const uint64_t m = __builtin_amdgcn_ballot_w64(cnt > 0);
    if (m) {
      const int lead = (int)__builtin_ctzll(m);
      const int d0 = __shfl(cur, lead, kWave);
      if (__builtin_amdgcn_ballot_w64(cnt > 0 && cur != d0) == 0) {
        const int tot = wave_sum_int(cnt);
        if (lane == lead) atomicAdd(&s_hist[wv][d0], tot);
      } else if (cnt > 0) {
        atomicAdd(&s_hist[wv][cur], cnt);
      }
    }
    __syncthreads();
    if (wv == 0) {
      // lane l holds digits 4l .. 4l + 3, lowest first
      int c[4], tot = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int h = 0;
        for (int q2 = 0; q2 < kPlanWaves; ++q2) h += s_hist[q2][4 * lane + i];
        c[i] = h;
        tot += h;
      }
      int incl = tot;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o, kWave);
        if (lane >= o) incl += y;
      }
      int cum = below + incl - tot;
      int hit_d = -1, before = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (hit_d < 0 && cum + c[i] >= k) {
          hit_d = 4 * lane + i;
          before = cum;
        }
        cum += c[i];
      }
      const uint64_t found = __builtin_amdgcn_ballot_w64(hit_d >= 0);
      const int all = __shfl(incl, 63, kWave);
      if (found && lane == (int)__builtin_ctzll(found)) {
        s_below = before;
        s_thr = (prefix << 8) | hit_d;
      } else if (!found && lane == 0) {
        // fewer than k candidates (only a stale slot_step leaves that): every
        // candidate is a victim, the threshold above them all
        s_below = below + all;
        s_thr = (prefix << 8) + 256;
      }
    }
    __syncthreads();
    below = s_below;
    prefix = s_thr;
  }
  // victims: keys below the threshold, then the first (k - below) slots with
  // the threshold key, in slot order; the q-th new row (selection order) goes
  // to the q-th victim (slot order)
  const int thr = prefix;
  const int take_eq = k - below;
  uint64_t victim = 0;
  int n_victims = 0, v_first = 0;
  if (k > 0) {
    int n_lt = 0, n_eq = 0;
#pragma unroll
    for (int j = 0; j < R; ++j) {
      n_lt += key[j] <= step && key[j] < thr;
      n_eq += key[j] <= step && key[j] == thr;
    }
    int eq_before;
    block_scan_count(n_eq, s_w, eq_before);
    int e = eq_before;
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const int x = key[j];
      if (x > step) continue;
      if (x < thr || (x == thr && e < take_eq)) victim |= 1ull << j;
      e += x == thr;
    }
    n_victims = block_scan_count(__popcll(victim), s_w, v_first);
#pragma unroll
    for (int j = 0, o = v_first; j < R; ++j)
      if (victim >> j & 1ull) {
        if (o < budget) fetch_slot[(size_t)s * budget + o] = i0 + j;
        ++o;
      }
  }
  n_victims = min(n_victims, budget);
  __syncthreads();
  // the new rows in selection order: the q-th takes victim q's slot (rows
  // beyond the victims, only possible with a stale slot_step, get none)
  int base = 0;
  const int prounds = (n + kPlanThreads - 1) / kPlanThreads;
  for (int rd = 0; rd < prounds; ++rd) {
    const int p = rd * kPlanThreads + tid;
    int r = -1;
    bool nw = false;
    if (p < n) {
      r = rows[p];
      nw = r >= 0 && r < pool_rows && (s_bits[r >> 5] >> (r & 31) & 1u);
    }
    int ex;
    const int tot = block_scan_flag(nw, s_w, ex);
    if (nw) {
      const int q = base + ex;
      const int slot = q < n_victims ? fetch_slot[(size_t)s * budget + q] : -1;
      fetch_row[(size_t)s * budget + q] = slot >= 0 ? r : -1;
      if (slot >= 0 && slot < cache_rows) {
        brow[slot] = r;
        bstep[slot] = step;
      }
    }
    base += tot;
  }
  if (tid == 0) {
    n_fetch[s] = k;
    if (n_fetch_out) n_fetch_out[s] = k;
  }
  // the slots that hold the selection, in slot order: hits and the victims
  // that took a new row
  uint64_t held = hit;
  {
    int o = v_first;
#pragma unroll
    for (int j = 0; j < R; ++j)
      if (victim >> j & 1ull) {
        if (o < min(k, n_victims)) held |= 1ull << j;
        ++o;
      }
  }
  int before;
  block_scan_count(__popcll(held), s_w, before);
#pragma unroll
  for (int j = 0, o = before; j < R; ++j)
    if (held >> j & 1ull) {
      if (o < budget) slot_list[(size_t)s * budget + o] = i0 + j;
      ++o;
    }
}

// Copy the planned rows pool -> buffer slot: 16 lanes per row, 16 rows per pass.
template <class T>
__global__ __launch_bounds__(256)
void delta_fetch_kernel(const T* __restrict__ k_pool, const T* __restrict__ v_pool, int64_t pool_rows,
                        const int32_t* __restrict__ fetch_slot, const int32_t* __restrict__ fetch_row,
                        const int32_t* __restrict__ n_fetch, int budget, int blocks_per_slice, int rows_per_block,
                        T* __restrict__ k_buf, T* __restrict__ v_buf, int buf_rows) {
  const int64_t s = blockIdx.x / blocks_per_slice;
  const int b = (int)(blockIdx.x - s * blocks_per_slice);
  const int n = n_fetch[s];
  const int r0 = b * rows_per_block;
  if (r0 >= n) return;
  const int r1 = min(n, r0 + rows_per_block);
  constexpr int kU4 = kHeadDim * sizeof(T) / 16;
  const int sub = threadIdx.x & 15;
  for (int k = r0 + (threadIdx.x >> 4); k < r1; k += 16) {
    const int64_t pr = fetch_row[(size_t)s * budget + k];
    const int slot = fetch_slot[(size_t)s * budget + k];
    if (pr < 0 || pr >= pool_rows || slot < 0 || slot >= buf_rows) continue;
    const uint4* ks = reinterpret_cast<const uint4*>(k_pool + ((size_t)s * pool_rows + pr) * kHeadDim);
    const uint4* vs = reinterpret_cast<const uint4*>(v_pool + ((size_t)s * pool_rows + pr) * kHeadDim);
    uint4* kd = reinterpret_cast<uint4*>(k_buf + ((size_t)s * buf_rows + slot) * kHeadDim);
    uint4* vd = reinterpret_cast<uint4*>(v_buf + ((size_t)s * buf_rows + slot) * kHeadDim);
#pragma unroll
    for (int q = sub; q < kU4; q += 16) {
      const uint4 a = ks[q], c = vs[q];
      kd[q] = a;
      vd[q] = c;
    }
  }
}

// ------------------------------------------------------------------ attention

// Zero-copy retrieval: the selected rows are read straight from the pool
// through the slice's row list.  A block copies its chunk's entries
// [lo, hi) of the list into LDS, clamped into the pool so that a malformed
// list cannot address memory outside it, and waits for the copy.
__device__ __forceinline__ void stage_row_list(const int32_t* __restrict__ list, int lo, int hi, int64_t src_rows,
                                               int* s_rows, int tid, int n_threads) {
  for (int i = lo + tid; i < hi; i += n_threads)
    s_rows[i - lo] = (int)min<int64_t>(max(list[i], 0), src_rows - 1);
  __syncthreads();
}

// Blocks of 8 waves (attn_mfma_waves; two fit a CU where a wave needs at
// most 128 VGPRs).  A slice's rows go to one block when there are enough
// slices to fill the chip; otherwise they are cut into n_chunks equal ranges
// (split-KV), never below kAttnMinRows rows per block, and a second kernel
// merges the chunk partials.
constexpr int kAttnTargetBlocks = 256;
constexpr int kAttnMinRows = 256;
// A fused decode step over few slices spreads each slice's rows over many
// small blocks: kStepAttnRows rows per block of kStepAttnWaves waves.
#ifndef LKV_STEP_ATTN_ROWS
#define LKV_STEP_ATTN_ROWS 128
#endif
constexpr int kStepAttnWaves = 8;
constexpr int kStepAttnRows = LKV_STEP_ATTN_ROWS;

// Sum over the 16 lanes of a DPP row, result in every lane of the row:
// butterflies over lane^1, lane^2 (quad permutes), then the mirrored halves
// of 8 and of 16 lanes.  All VALU, no LDS traffic.
__device__ __forceinline__ float row16_sum(float x) {
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0xB1, 0xF, 0xF, false));
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x4E, 0xF, 0xF, false));
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x141, 0xF, 0xF, false));
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x140, 0xF, 0xF, false));
  return x;
}

constexpr float kLog2e = 1.4426950408889634f;

// One lane's share (8 dims) of a K or V row, kept in storage format until used.
template <class T> struct Raw8;
template <> struct Raw8<uint16_t> {
  uint32_t w[4];
  __device__ __forceinline__ void load(const uint16_t* p) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
  }
  __device__ __forceinline__ float at(int e) const {
    return __uint_as_float((e & 1) ? (w[e >> 1] & 0xffff0000u) : (w[e >> 1] << 16));
  }
  // sum_e a[e] * this[e] with fp32 accumulation of the exact bf16 products
  __device__ __forceinline__ float dot(const Raw8& a) const {
    typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
    float d = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      d = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf2, a.w[i]), __builtin_bit_cast(bf2, w[i]), d, false);
    return d;
  }
};
template <> struct Raw8<float> {
  float x[8];
  __device__ __forceinline__ void load(const float* p) {
    const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
  }
  __device__ __forceinline__ float at(int e) const { return x[e]; }
  __device__ __forceinline__ float dot(const Raw8& a) const {
    float d = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) d = fmaf(a.x[e], x[e], d);
    return d;
  }
};

// Rows each 16-lane group keeps in flight: enough loads outstanding to cover
// HBM latency at the occupancy the register footprint allows.
template <class T, int G>
constexpr int attn_rows_in_flight() {
  return (sizeof(T) == 2 ? 4 : 2) / (G == 8 ? 2 : 1);
}
template <class T, int G>
constexpr int attn_waves() {
  return sizeof(T) == 2 && G <= 4 ? 16 : 8;
}

// What the attention blocks of a fused decode step do beyond the attention:
// with `counter` (per-slice arrival counters, zero between calls) a slice's
// chunk partials are merged by its last block to finish instead of by
// attn_combine_kernel, and with `q_ref` one block per group stores the
// step's query as the new reference (every step in PREV mode, at a fire in
// ANCHOR mode) once the boundary test has read the old one.
struct StepSync {
  int32_t* counter;
  void* q_ref;
  const uint8_t* fire;
  int mode;
};

template <class T>
__device__ __forceinline__ void update_q_ref(const StepSync& sync, const T* __restrict__ q, int64_t grp, int n_elems,
                                             int tid, int n_threads) {
  if (!(sync.mode == LOUISKV_REF_PREV || sync.fire[grp])) return;
  T* dst = static_cast<T*>(sync.q_ref) + (size_t)grp * n_elems;
  const T* src = q + (size_t)grp * n_elems;
  for (int i = tid; i < n_elems; i += n_threads) dst[i] = src[i];
}

// The last of a slice's n_chunks blocks to arrive merges their partials,
// (m, l, acc[128]) per head in base 2, in chunk order with the arithmetic of
// attn_combine_kernel, so the outputs equal the two-kernel path's bit for bit.
// Partials are written and read with device-scope atomic stores and loads
// (coherent across the per-XCD L2 caches); a block waits for its stores
// before it counts itself in, and the last one resets the counter.  The
// merging block first stages every chunk's (m, l) in LDS (s_ml, n_chunks * G
// pairs), then each thread takes one head and two dims and reads their
// accumulators kMergeBatch chunks at a time, all loads of a batch in flight.
constexpr int kMergeBatch = 32;

template <int G, bool kOneTrip = false>
__device__ __forceinline__ bool attn_last_block_merge(const float* __restrict__ part, int32_t* __restrict__ counter,
                                                      int64_t s, int n_chunks, void* __restrict__ out, int out_bf16,
                                                      float* __restrict__ lse_out, int tid, int n_threads,
                                                      float2* s_ml) {
  __shared__ int s_last;
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (tid == 0) {
    const int old = __hip_atomic_fetch_add(counter, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_last = old == n_chunks - 1;
    if (s_last) __hip_atomic_store(counter, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (!s_last) return false;
  constexpr size_t pstride = 2 + kHeadDim;
  const float* ps = part + (size_t)s * n_chunks * G * pstride;
  if (kOneTrip && n_chunks <= kMergeBatch) {
    // every chunk's (m, l) and accumulators of a thread's head and two dims
    // loaded at once: one round trip, the same arithmetic as below
    for (int i = tid; i < G * (kHeadDim / 2); i += n_threads) {
      const int j = i / (kHeadDim / 2), lane = i % (kHeadDim / 2);
      const uint64_t* pm = reinterpret_cast<const uint64_t*>(ps + (size_t)j * pstride);
      const uint64_t* pa = reinterpret_cast<const uint64_t*>(ps + (size_t)j * pstride + 2) + lane;
      uint64_t mlv[kMergeBatch], v[kMergeBatch];
#pragma unroll
      for (int c = 0; c < kMergeBatch; ++c) {
        mlv[c] = c < n_chunks ? __hip_atomic_load(pm + (size_t)c * G * (pstride / 2), __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT)
                              : 0;
        v[c] = c < n_chunks ? __hip_atomic_load(pa + (size_t)c * G * (pstride / 2), __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT)
                            : 0;
      }
      float mm = -__builtin_inff();
#pragma unroll
      for (int c = 0; c < kMergeBatch; ++c)
        if (c < n_chunks) mm = fmaxf(mm, __uint_as_float((uint32_t)mlv[c]));
      float ll = 0.f, a0 = 0.f, a1 = 0.f;
      if (mm != -__builtin_inff()) {
#pragma unroll
        for (int c = 0; c < kMergeBatch; ++c) {
          if (c < n_chunks) {
            const float w = __builtin_amdgcn_exp2f(__uint_as_float((uint32_t)mlv[c]) - mm);
            ll += __uint_as_float((uint32_t)(mlv[c] >> 32)) * w;
            a0 += __uint_as_float((uint32_t)v[c]) * w;
            a1 += __uint_as_float((uint32_t)(v[c] >> 32)) * w;
          }
        }
      }
      const float inv = ll > 0.f ? 1.f / ll : 0.f;
      const size_t row = (size_t)s * G + j;
      if (out_bf16) {
        uint16_t* o = static_cast<uint16_t*>(out) + row * kHeadDim;
        store_from_f32(o, 2 * lane, a0 * inv);
        store_from_f32(o, 2 * lane + 1, a1 * inv);
      } else {
        float* o = static_cast<float*>(out) + row * kHeadDim;
        store_from_f32(o, 2 * lane, a0 * inv);
        store_from_f32(o, 2 * lane + 1, a1 * inv);
      }
      if (lse_out && lane == 0) lse_out[row] = ll > 0.f ? 0.6931471805599453f * (mm + log2f(ll)) : -__builtin_inff();
    }
    return true;
  }
  for (int i = tid; i < n_chunks * G; i += n_threads) {
    const uint64_t v = __hip_atomic_load(reinterpret_cast<const uint64_t*>(ps + (size_t)i * pstride),
                                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_ml[i] = make_float2(__uint_as_float((uint32_t)v), __uint_as_float((uint32_t)(v >> 32)));
  }
  __syncthreads();
  for (int i = tid; i < G * (kHeadDim / 2); i += n_threads) {
    const int j = i / (kHeadDim / 2), lane = i % (kHeadDim / 2);
    float mm = -__builtin_inff();
    for (int c = 0; c < n_chunks; ++c) mm = fmaxf(mm, s_ml[c * G + j].x);
    float ll = 0.f, a0 = 0.f, a1 = 0.f;
    if (mm != -__builtin_inff()) {
      const uint64_t* pa = reinterpret_cast<const uint64_t*>(ps + (size_t)j * pstride + 2) + lane;
      for (int c0 = 0; c0 < n_chunks; c0 += kMergeBatch) {
        uint64_t v[kMergeBatch];
#pragma unroll
        for (int b = 0; b < kMergeBatch; ++b)
          v[b] = c0 + b < n_chunks ? __hip_atomic_load(pa + (size_t)(c0 + b) * G * (pstride / 2), __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT)
                                   : 0;
#pragma unroll
        for (int b = 0; b < kMergeBatch; ++b) {
          if (c0 + b < n_chunks) {
            const float2 ml = s_ml[(c0 + b) * G + j];
            const float w = __builtin_amdgcn_exp2f(ml.x - mm);
            ll += ml.y * w;
            a0 += __uint_as_float((uint32_t)v[b]) * w;
            a1 += __uint_as_float((uint32_t)(v[b] >> 32)) * w;
          }
        }
      }
    }
    const float inv = ll > 0.f ? 1.f / ll : 0.f;
    const size_t row = (size_t)s * G + j;
    if (out_bf16) {
      uint16_t* o = static_cast<uint16_t*>(out) + row * kHeadDim;
      store_from_f32(o, 2 * lane, a0 * inv);
      store_from_f32(o, 2 * lane + 1, a1 * inv);
    } else {
      float* o = static_cast<float*>(out) + row * kHeadDim;
      store_from_f32(o, 2 * lane, a0 * inv);
      store_from_f32(o, 2 * lane + 1, a1 * inv);
    }
    if (lse_out && lane == 0) lse_out[row] = ll > 0.f ? 0.6931471805599453f * (mm + log2f(ll)) : -__builtin_inff();
  }
  return true;
}

// Merge NW wave states (base-2 maximum m and sum l per head, acc per head and
// dim, all in LDS) into the block's result: the normalised output and lse when
// the block covers the whole slice (n_chunks == 1), else the chunk partial
// (m, l, acc[128]) per head for attn_combine_kernel, or, with `counter` (the
// slice's arrival counter), for the in-kernel merge.  True when this block
// wrote the slice's output (one chunk, or the last block of an in-kernel merge).
template <int G, int NW, bool kOneTrip = false>
__device__ __forceinline__ bool attn_block_merge(const float (*s_m)[G], const float (*s_l)[G],
                                                 const float (*s_acc)[G][kHeadDim], int tid, int64_t s, int chunk,
                                                 int n_chunks, float* __restrict__ part, void* __restrict__ out,
                                                 int out_bf16, float* __restrict__ lse_out,
                                                 int32_t* __restrict__ counter, float2* s_ml) {
  for (int i = tid; i < G * kHeadDim; i += NW * 64) {
    const int j = i / kHeadDim, k = i % kHeadDim;
    float mm = -__builtin_inff();
    for (int q2 = 0; q2 < NW; ++q2) mm = fmaxf(mm, s_m[q2][j]);
    float ll = 0.f, aa = 0.f;
    if (mm != -__builtin_inff()) {
      for (int q2 = 0; q2 < NW; ++q2) {
        const float c = __builtin_amdgcn_exp2f(s_m[q2][j] - mm);
        ll += s_l[q2][j] * c;
        aa += s_acc[q2][j][k] * c;
      }
    }
    if (n_chunks == 1) {
      const size_t row = (size_t)s * G + j;    // (group, query head) row of the output
      const float o = ll > 0.f ? aa / ll : 0.f;
      if (out_bf16)
        static_cast<uint16_t*>(out)[row * kHeadDim + k] = f32_to_bf16(o);
      else
        static_cast<float*>(out)[row * kHeadDim + k] = o;
      // base-2 maxima: lse = ln 2 * (m + log2 l)
      if (lse_out && k == 0) lse_out[row] = ll > 0.f ? 0.6931471805599453f * (mm + log2f(ll)) : -__builtin_inff();
    } else {
      const size_t pstride = 2 + kHeadDim;
      float* pout = part + ((size_t)s * n_chunks + chunk) * G * pstride;
      if (counter) {   // read back by another block of this launch
        __hip_atomic_store(pout + j * pstride + 2 + k, aa, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (k == 0) {
          __hip_atomic_store(pout + j * pstride + 0, mm, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_store(pout + j * pstride + 1, ll, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      } else {
        pout[j * pstride + 2 + k] = aa;
        if (k == 0) {
          pout[j * pstride + 0] = mm;
          pout[j * pstride + 1] = ll;
        }
      }
    }
  }
  if (n_chunks == 1) return true;
  if (counter)
    return attn_last_block_merge<G, kOneTrip>(part, counter, s, n_chunks, out, out_bf16, lse_out, tid, NW * 64, s_ml);
  return false;
}

// With boundary-delimited segments the window of slice s holds the tokens
// from its first token (state) to n_tokens - 1; otherwise the arguments hold.
__device__ __forceinline__ void slice_window(const int32_t* seg_state, int seg_stride, int64_t s, int window,
                                             int n_tokens, int& local_start, int& n_local) {
  if (!seg_state) return;
  const int wf = seg_state[s * seg_stride + kSegWinFirst];
  n_local = min(max(n_tokens - wf, 0), window);
  local_start = wf >= 0 ? wf % window : 0;
}

// Block (chunk, slice): online softmax over the chunk's share of rows for the G
// query heads of the slice, in base 2 (logits scaled by log2 e / sqrt d);
// 16 lanes per row, lane sub owns dims 8*sub..+7, and each of the 64 row groups
// takes every 64th row, R rows per pass with all their loads issued up front.
// The running maximum and the rescale of the accumulators change only when
// some lane's maximum grows (a wave-uniform branch with per-lane selects).
// With one chunk the block writes the normalised output (and lse); otherwise
// it writes (m, l, acc[128]) per head, m in base 2, for the merge kernel.
template <class T, int G, bool kIdx>
__global__ __launch_bounds__((attn_waves<T, G>() * 64))
void attn_partial_kernel(const T* __restrict__ q, int n_kv_heads, float scale, const T* __restrict__ k_buf,
                         const T* __restrict__ v_buf, const int32_t* __restrict__ n_sel, int buf_rows,
                         const int32_t* __restrict__ rows, int64_t src_rows,
                         const T* __restrict__ k_local, const T* __restrict__ v_local, int window, int local_start_arg,
                         int n_local_arg, int n_chunks, float* __restrict__ part, void* __restrict__ out, int out_bf16,
                         float* __restrict__ lse_out, const int32_t* __restrict__ seg_state, int seg_stride,
                         int n_tokens, int slice_div, StepSync sync) {
  extern __shared__ __align__(16) int s_rows[];   // kIdx: the chunk's entries of the row list
  constexpr int R = attn_rows_in_flight<T, G>();
  constexpr int kAttnWaves = attn_waves<T, G>();
  constexpr int kAttnThreads = kAttnWaves * 64;
  constexpr int kAttnGroups = kAttnWaves * 4;      // 16-lane row groups per block
  __shared__ float s_m[kAttnWaves][G], s_l[kAttnWaves][G];
  __shared__ float s_acc[kAttnWaves][G][kHeadDim];
  const int64_t s = blockIdx.x / n_chunks;
  const int chunk = (int)(blockIdx.x - s * n_chunks);
  const int64_t grp = s / n_kv_heads;
  const int kvh = (int)(s - grp * n_kv_heads);
  const int tid = threadIdx.x, sub = tid & 15, rg = tid >> 4;   // 64 row groups of 16 lanes
  if (sync.q_ref && chunk == 0 && kvh == 0) update_q_ref(sync, q, grp, n_kv_heads * G * kHeadDim, tid, kAttnThreads);
  int local_start = local_start_arg, n_local = n_local_arg;
  // slice_div > 1: per-head lists, s is a query head and ps its KV head's slice
  const int64_t ps = s / slice_div;
  slice_window(seg_state, seg_stride, ps, window, n_tokens, local_start, n_local);
  const int nsel = max(0, min(n_sel[s], buf_rows));
  const int total = nsel + n_local;
  const int r0 = (int)((int64_t)total * chunk / n_chunks);
  const int r1 = (int)((int64_t)total * (chunk + 1) / n_chunks);
  const int n_pass = r1 > r0 ? (r1 - r0 + kAttnGroups * R - 1) / (kAttnGroups * R) : 0;   // block-uniform

  Raw8<T> qv[G];
  const size_t qbase = ((size_t)grp * n_kv_heads * G + (size_t)kvh * G) * kHeadDim + 8 * sub;
#pragma unroll
  for (int j = 0; j < G; ++j) qv[j].load(q + qbase + (size_t)j * kHeadDim);
  const float qs = scale * kLog2e;
  float m[G], l[G], acc[G][8];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    m[j] = -__builtin_inff();
    l[j] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[j][e] = 0.f;
  }
  const T* kb = k_buf + (size_t)ps * src_rows * kHeadDim + 8 * sub;
  const T* vb = v_buf + (size_t)ps * src_rows * kHeadDim + 8 * sub;
  const T* kl = k_local + (size_t)ps * window * kHeadDim + 8 * sub;
  const T* vl = v_local + (size_t)ps * window * kHeadDim + 8 * sub;
  if (kIdx) stage_row_list(rows + (size_t)s * buf_rows, r0, min(r1, nsel), src_rows, s_rows, tid, kAttnThreads);
  // Issue the loads of pass ps; rows past the chunk re-read its first row and
  // are masked.
  auto load_pass = [&](int ps, Raw8<T>* kx, Raw8<T>* vx, bool* valid) {
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const int r = r0 + rg + kAttnGroups * (ps * R + i);
      valid[i] = r < r1;
      const int rr = valid[i] ? r : r0;
      size_t off;
      const T* kp;
      const T* vp;
      if (rr < nsel) {
        off = (size_t)(kIdx ? s_rows[rr - r0] : rr) * kHeadDim;
        kp = kb; vp = vb;
      } else {
        int slot = local_start + (rr - nsel);      // local_start < window and rr - nsel < n_local <= window
        slot -= slot >= window ? window : 0;
        off = (size_t)slot * kHeadDim;
        kp = kl; vp = vl;
      }
      kx[i].load(kp + off);
      vx[i].load(vp + off);
    }
  };
  auto compute_pass = [&](const Raw8<T>* kx, const Raw8<T>* vx, const bool* valid) {
    float sc[R][G];
    bool grow = false;
#pragma unroll
    for (int i = 0; i < R; ++i) {
#pragma unroll
      for (int j = 0; j < G; ++j) {
        const float d = row16_sum(kx[i].dot(qv[j])) * qs;
        sc[i][j] = valid[i] ? d : -__builtin_inff();
        grow |= sc[i][j] > m[j];
      }
    }
    // rescale only when some lane's running maximum grows
    if (__builtin_amdgcn_ballot_w64(grow)) {
#pragma unroll
      for (int j = 0; j < G; ++j) {
        float mn = m[j];
#pragma unroll
        for (int i = 0; i < R; ++i) mn = fmaxf(mn, sc[i][j]);
        const float corr = mn == -__builtin_inff() ? 1.f : __builtin_amdgcn_exp2f(m[j] - mn);
        l[j] *= corr;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[j][e] *= corr;
        m[j] = mn;
      }
    }
#pragma unroll
    for (int i = 0; i < R; ++i) {
#pragma unroll
      for (int j = 0; j < G; ++j) {
        const float p = valid[i] ? __builtin_amdgcn_exp2f(sc[i][j] - m[j]) : 0.f;
        l[j] += p;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[j][e] = fmaf(p, vx[i].at(e), acc[j][e]);
      }
    }
  };
  for (int ps = 0; ps < n_pass; ++ps) {
    Raw8<T> kx[R], vx[R];
    bool valid[R];
    load_pass(ps, kx, vx, valid);
    __builtin_amdgcn_sched_barrier(0);   // keep every load of the pass ahead of its first use
    compute_pass(kx, vx, valid);
  }
  // merge the 4 row groups of each wave (lanes l, l^16, l^32, l^48 share sub)
#pragma unroll
  for (int j = 0; j < G; ++j) {
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      const float mo = __shfl_xor(m[j], o, kWave);
      const float lo = __shfl_xor(l[j], o, kWave);
      const float mn = fmaxf(m[j], mo);
      const float ca = mn == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(m[j] - mn);
      const float cb = mn == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(mo - mn);
      l[j] = l[j] * ca + lo * cb;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float ao = __shfl_xor(acc[j][e], o, kWave);
        acc[j][e] = acc[j][e] * ca + ao * cb;
      }
      m[j] = mn;
    }
  }
  const int w = tid >> 6;
  if ((tid & 63) < 16) {
#pragma unroll
    for (int j = 0; j < G; ++j) {
      if (sub == 0) {
        s_m[w][j] = m[j];
        s_l[w][j] = l[j];
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) s_acc[w][j][8 * sub + e] = acc[j][e];
    }
  }
  __syncthreads();
  attn_block_merge<G, kAttnWaves>(s_m, s_l, s_acc, tid, s, chunk, n_chunks, part, out, out_bf16, lse_out,
                                  sync.counter ? sync.counter + s : nullptr, reinterpret_cast<float2*>(s_rows));
}

// ---- bf16: scores on the matrix cores

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 attn_bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float attn_floatx4;

__device__ __forceinline__ float row16_max(float x) {
  x = fmaxf(x, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0xB1, 0xF, 0xF, false)));
  x = fmaxf(x, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x4E, 0xF, 0xF, false)));
  x = fmaxf(x, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x141, 0xF, 0xF, false)));
  x = fmaxf(x, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x140, 0xF, 0xF, false)));
  return x;
}

// Waves per attention block: 8 for every group size.  With one block per
// slice, 8-wave blocks were 3-6% faster than 16-wave ones on 256 slices (a
// shorter in-block merge of the waves' partials; 8 waves keep enough rows in
// flight) and as fast on 1024.
template <int G>
constexpr int attn_mfma_waves() {
  return 8;
}

// The A operand of the score MFMAs from the slice's G query rows (qs): row
// m = l%16 of op mi holds head 4*mi + m % min(G, 4); k-chunk c covers dims
// 32c..32c+31.
template <int G, int NM = (G == 8 ? 2 : 1)>
__device__ __forceinline__ void load_attn_q(const uint16_t* __restrict__ qs, int lane, attn_bf16x8 (&qa)[NM][4]) {
  constexpr int GA = G < 4 ? G : 4;
  const int g = lane >> 4, p16 = lane & 15;
#pragma unroll
  for (int mi = 0; mi < NM; ++mi)
#pragma unroll
    for (int c = 0; c < 4; ++c)
      qa[mi][c] = __builtin_bit_cast(
          attn_bf16x8, *reinterpret_cast<const uint4*>(qs + (size_t)(4 * mi + p16 % GA) * kHeadDim + 32 * c + 8 * g));
}

// One 16-row tile of a wave: the scores of the tile's K rows (kx: lane l
// holds row l%16) from v_mfma_f32_16x16x32_bf16, the base-2 online softmax
// update of (m, l, acc) and P V with the tile's V rows (vx: rows 4k + l/16,
// dims 8(l%16)..+7).  s_pw is the wave's LDS slot for the probabilities.
template <int G, int NM = (G == 8 ? 2 : 1)>
__device__ __forceinline__ void attn_mfma_tile(const attn_bf16x8 (&qa)[NM][4], const uint4 (&kx)[4],
                                               const uint4 (&vx)[4], bool kvalid, float qscale, float (&m)[G],
                                               float (&l)[G], float (&acc)[G][8], float4 (*s_pw)[64], int lane) {
  const int g = lane >> 4;
  __builtin_amdgcn_sched_barrier(0);   // keep the tile's loads ahead of their first use
  attn_floatx4 sacc[NM];
#pragma unroll
  for (int mi = 0; mi < NM; ++mi) {
    sacc[mi] = attn_floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < 4; ++c)
      sacc[mi] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[mi][c], __builtin_bit_cast(attn_bf16x8, kx[c]), sacc[mi],
                                                        0, 0, 0);
  }
  float sc[G];
  bool grow = false;
#pragma unroll
  for (int j = 0; j < G; ++j) {
    const float x = sacc[j / 4][j % 4] * qscale;    // head j of row kr (regs i >= GA repeat heads)
    sc[j] = kvalid ? x : -__builtin_inff();
    grow |= sc[j] > m[j];
  }
  // rescale only when some row's score exceeds its head's running maximum
  if (__builtin_amdgcn_ballot_w64(grow)) {
#pragma unroll
    for (int j = 0; j < G; ++j) {
      const float mn = fmaxf(m[j], row16_max(sc[j]));
      const float corr = mn == -__builtin_inff() ? 1.f : __builtin_amdgcn_exp2f(m[j] - mn);
      l[j] *= corr;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[j][e] *= corr;
      m[j] = mn;
    }
  }
  float pr[NM * 4];
#pragma unroll
  for (int j = 0; j < NM * 4; ++j) pr[j] = 0.f;
#pragma unroll
  for (int j = 0; j < G; ++j) {
    pr[j] = kvalid ? __builtin_amdgcn_exp2f(sc[j] - m[j]) : 0.f;
    l[j] += pr[j];
  }
  // probabilities of row p16 to the lanes that hold its V row
#pragma unroll
  for (int mi = 0; mi < NM; ++mi)
    s_pw[mi][lane] = make_float4(pr[4 * mi], pr[4 * mi + 1], pr[4 * mi + 2], pr[4 * mi + 3]);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    float pk[NM * 4];
#pragma unroll
    for (int mi = 0; mi < NM; ++mi) {
      const float4 f = s_pw[mi][4 * k + g + 16 * g];
      pk[4 * mi] = f.x; pk[4 * mi + 1] = f.y; pk[4 * mi + 2] = f.z; pk[4 * mi + 3] = f.w;
    }
    float vf[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t wv = (&vx[k].x)[i];
      vf[2 * i] = __uint_as_float(wv << 16);
      vf[2 * i + 1] = __uint_as_float(wv & 0xffff0000u);
    }
#pragma unroll
    for (int j = 0; j < G; ++j)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[j][e] = fmaf(pk[j], vf[e], acc[j][e]);
  }
}

// A wave's totals into its LDS slot: l over the 16 row positions, acc over
// the 4 lane groups (m is wave-uniform).
template <int G>
__device__ __forceinline__ void attn_wave_to_lds(const float (&m)[G], float (&l)[G], float (&acc)[G][8], float* s_mw,
                                                 float* s_lw, float (*s_accw)[kHeadDim], int lane) {
#pragma unroll
  for (int j = 0; j < G; ++j) {
    l[j] = row16_sum(l[j]);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      acc[j][e] += __shfl_xor(acc[j][e], 16, kWave);
      acc[j][e] += __shfl_xor(acc[j][e], 32, kWave);
    }
  }
  if (lane < 16) {
#pragma unroll
    for (int j = 0; j < G; ++j) {
      if (lane == 0) {
        s_mw[j] = m[j];
        s_lw[j] = l[j];
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) s_accw[j][8 * lane + e] = acc[j][e];
    }
  }
}

// Block (chunk, slice) for bf16 K/V.  A wave takes 16-row tiles t = w, w+NW, ...
// of the chunk.  Scores S = Q K^T come from v_mfma_f32_16x16x32_bf16 with the
// tile's K rows as the B operand (lane l: row l%16, dims 32c+8(l/16)..+7 of
// k-chunk c) and Q as the A operand, its g heads repeated over the 16 rows of
// A, so that every lane receives the scores of its row (l%16) for all heads.
// The base-2 online softmax runs per lane on those scores; the probabilities
// go through a per-wave LDS slot to the V layout of the PV step, 16 lanes per
// row (lane owns dims 8(l%16)..+7, rows 4k + l/16 of the tile for k = 0..3),
// where P V accumulates in float32 on the vector ALUs.  Output and partials as
// attn_partial_kernel.
template <int G, bool kIdx, int NW = attn_mfma_waves<G>()>
__global__ __launch_bounds__((NW * 64))
void attn_mfma_kernel(const uint16_t* __restrict__ q, int n_kv_heads, float scale, const uint16_t* __restrict__ k_buf,
                      const uint16_t* __restrict__ v_buf, const int32_t* __restrict__ n_sel, int buf_rows,
                      const int32_t* __restrict__ rows, int64_t src_rows,
                      const uint16_t* __restrict__ k_local, const uint16_t* __restrict__ v_local, int window,
                      int local_start_arg, int n_local_arg, int n_chunks, float* __restrict__ part,
                      void* __restrict__ out, int out_bf16, float* __restrict__ lse_out,
                      const int32_t* __restrict__ seg_state, int seg_stride, int n_tokens, int slice_div,
                      StepSync sync) {
  extern __shared__ __align__(16) int s_rows[];   // kIdx: the chunk's entries of the row list
  constexpr int NM = G == 8 ? 2 : 1;        // matrix ops per k-chunk, 4 heads each
  __shared__ float4 s_p[NW][NM][64];
  __shared__ float s_m[NW][G], s_l[NW][G];
  __shared__ float s_acc[NW][G][kHeadDim];
  const int64_t s = blockIdx.x / n_chunks;
  const int chunk = (int)(blockIdx.x - s * n_chunks);
  const int64_t grp = s / n_kv_heads;
  const int kvh = (int)(s - grp * n_kv_heads);
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 4, p16 = lane & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);    // wave-uniform, kept in a scalar register
  if (sync.q_ref && chunk == 0 && kvh == 0) update_q_ref(sync, q, grp, n_kv_heads * G * kHeadDim, tid, NW * 64);
  int local_start = local_start_arg, n_local = n_local_arg;
  // slice_div > 1: per-head lists, s is a query head and ps its KV head's slice
  const int64_t ps = s / slice_div;
  slice_window(seg_state, seg_stride, ps, window, n_tokens, local_start, n_local);
  const int nsel = max(0, min(n_sel[s], buf_rows));
  const int total = nsel + n_local;
  const int r0 = (int)((int64_t)total * chunk / n_chunks);
  const int r1 = (int)((int64_t)total * (chunk + 1) / n_chunks);
  const int n_tiles = (r1 - r0 + 15) / 16;   // block-uniform

  attn_bf16x8 qa[NM][4];
  load_attn_q<G>(q + ((size_t)grp * n_kv_heads + kvh) * G * kHeadDim, lane, qa);
  const float qscale = scale * kLog2e;
  float m[G], l[G], acc[G][8];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    m[j] = -__builtin_inff();
    l[j] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[j][e] = 0.f;
  }
  const uint16_t* kb = k_buf + (size_t)ps * src_rows * kHeadDim;
  const uint16_t* vb = v_buf + (size_t)ps * src_rows * kHeadDim;
  const uint16_t* kl = k_local + (size_t)ps * window * kHeadDim;
  const uint16_t* vl = v_local + (size_t)ps * window * kHeadDim;
  if (kIdx) stage_row_list(rows + (size_t)s * buf_rows, r0, min(r1, nsel), src_rows, s_rows, tid, NW * 64);
  // element offset of row r (valid) in its region, and which region
  auto row_off = [&](int r, bool& local) -> size_t {
    local = r >= nsel;
    int slot = local_start + (r - nsel);        // local_start < window and r - nsel < n_local <= window
    slot -= slot >= window ? window : 0;
    const int sel = kIdx ? s_rows[max(0, min(r, nsel - 1) - r0)] : r;   // index stays inside the staged chunk
    return (size_t)(local ? slot : sel) * kHeadDim;
  };

  for (int t = w; t < n_tiles; t += NW) {
    const int tb = r0 + 16 * t;
    // K rows for the B operand; rows past the chunk re-read its first row and are masked
    const int kr = tb + p16;
    const bool kvalid = kr < r1;
    bool kloc;
    const size_t koff = row_off(kvalid ? kr : r0, kloc);
    const uint16_t* kp = (kloc ? kl : kb) + koff + 8 * g;
    uint4 kx[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) kx[c] = *reinterpret_cast<const uint4*>(kp + 32 * c);
    uint4 vx[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int vr = tb + 4 * k + g;
      bool vloc;
      const size_t voff = row_off(vr < r1 ? vr : r0, vloc);
      vx[k] = *reinterpret_cast<const uint4*>((vloc ? vl : vb) + voff + 8 * p16);
    }
    attn_mfma_tile<G>(qa, kx, vx, kvalid, qscale, m, l, acc, s_p[w], lane);
  }
  attn_wave_to_lds<G>(m, l, acc, s_m[w], s_l[w], s_acc[w], lane);
  __syncthreads();
  attn_block_merge<G, NW>(s_m, s_l, s_acc, tid, s, chunk, n_chunks, part, out, out_bf16, lse_out,
                          sync.counter ? sync.counter + s : nullptr, reinterpret_cast<float2*>(s_rows));
}

// ---------------------------------------------------------------------------
// A bf16 decode step over few slices in one launch: n_blk blocks per slice,
// every one of which does a part of the retrieval and a chunk of the
// attention, so that a layer's few slices spread over the whole chip.
//
// Block c of slice s computes r (the same float64 value in every block of
// the group) while it loads its chunk's entries of the row list of the last
// fire, the list length and its Q operand; block 0 runs the fixed-segment
// store.  If the group fired, the block computes the logits of its part of
// the units and counts itself in (select_part): the last block to arrive
// makes the selection, writes the row list with device-scope stores and
// raises the slice's ready flag; the others wait for the flag and read the
// new list entries coherently.  Only blocks that have arrived wait, and they
// wait for the last arrival, which is running and waits for nothing; so the
// wait ends once every block of the slice has started, which holds when the
// whole grid is resident at once (the launch gives the chip at most one
// block per compute unit) and also when it is not, since workgroups are
// dispatched in index order and a slice's blocks are consecutive.  The wait
// is bounded all the same: past spin_limit polls (kStepSpinLimit, or fewer
// from LOUISKV_STEP_SPIN_LIMIT, for tests of this path) a block records a
// time-out in the status word and goes on; its row-list entries are clamped
// into the pool, so that such a step reads no memory out of bounds.  Then the block attends its chunk of the slice's row sequence (the
// selected rows, padded to the budget, then the window rows), two 16-row
// tiles per wave in flight; the newest window row is read from k_new/v_new,
// since the store of the same launch may not have reached the ring yet.  The
// last block of a slice to finish merges the chunk partials, and lowers the
// ready flag after a fire.
//
// Every block counts itself in at its group's counter once it has read q_ref;
// the last to arrive stores the new reference query (every step in PREV mode,
// at a fire in ANCHOR mode) and resets the counter, so that counters and flags
// are zero between calls.
constexpr int kStepSpinLimit = 1 << 20;
// Counters and flags of the fused step sit kStepSyncStride ints apart, each
// in a 256-byte block of its own: atomics on one line serialise.
constexpr int kStepSyncStride = 64;
// Blocks per slice: at most the one-trip merge's chunk count.
constexpr int kStepMaxBlocks = kMergeBatch;
static_assert(kStepMaxBlocks <= kMaxSelectParts, "a selection part per block");
// List entries a thread loads before it knows whether the group fired.
constexpr int kStepListEarly = 2;

struct FusedStep {
  const uint16_t* q;
  uint16_t* q_ref;
  int64_t n_slices;
  int n_kv_heads, first, mode;
  double tau;
  double* r_out;
  uint8_t* fire_out;
  const uint16_t *k_new, *v_new;
  uint16_t *k_local, *v_local;
  int window, step, seg_len, evict_seg;
  float* reps;
  int32_t *unit_start, *unit_size;
  int units_cap, n_clusters;
  uint16_t *k_pool, *v_pool;
  int64_t pool_rows;
  int prompt_len;
  double scale;
  int n_units, budget;
  int32_t *sel_units, *n_sel_units, *n_sel, *sel_rows;
  double* scores_out;
  double *logit_ws, *part_max;
  int32_t *sel_counter, *attn_counter, *ready, *grp_counter, *status;
  int n_blk, chunk_rows, n_pad, spin_limit;
  int local_start, n_local;
  float* part;
  void* out;
  int out_bf16;
  float* lse_out;
};

// LDS of the attention part of the fused step: wave probability slots,
// per-wave (m, l, acc), the merge's (m, l) pairs and the chunk's list entries.
template <int G>
constexpr size_t fused_attn_lds(int n_blk, int chunk_rows) {
  constexpr int NM = G == 8 ? 2 : 1;
  return (size_t)kSelWaves * NM * 64 * sizeof(float4) + (size_t)2 * kSelWaves * G * sizeof(float) +
         (size_t)kSelWaves * G * kHeadDim * sizeof(float) + (size_t)n_blk * G * sizeof(float2) +
         (size_t)chunk_rows * sizeof(int);
}

template <int G>
__global__ __launch_bounds__(kSelThreads)
void step_fused_kernel(const FusedStep a) {
  constexpr int NW = kSelWaves;
  constexpr int NM = G == 8 ? 2 : 1;
  extern __shared__ __align__(16) char smem[];
  __shared__ double s_bpart[16];
  __shared__ int s_grp_last;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 4, p16 = lane & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nb = a.n_blk;
  const int64_t s = blockIdx.x / nb;
  const int c = (int)(blockIdx.x - s * nb);
  const int64_t grp = s / a.n_kv_heads;
  const int kvh = (int)(s - grp * a.n_kv_heads);
  const int n_q_heads = a.n_kv_heads * G;
  // the chunk: positions [p0, p1) of the slice's row sequence, the selected
  // ones [p0, sel_hi)
  const int p0 = c * a.chunk_rows;
  const int p1 = max(p0, min(p0 + a.chunk_rows, a.budget + a.n_local));
  const int sel_hi = max(p0, min(p1, a.budget));
  const int32_t* rl = a.sel_rows + (size_t)s * a.budget;

  // the list of the last fire, its length and the Q operand, loaded with the
  // boundary test's inputs (every access to the list and its length is a
  // device-scope load: selecting blocks of this launch write them on a fire)
  int early[kStepListEarly];
#pragma unroll
  for (int e = 0; e < kStepListEarly; ++e) {
    const int i = tid + e * kSelThreads;
    early[e] = p0 + i < sel_hi ? __hip_atomic_load(rl + p0 + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
  }
  int nsel = __hip_atomic_load(a.n_sel + s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  attn_bf16x8 qa[NM][4];
  load_attn_q<G>(a.q + (size_t)s * G * kHeadDim, lane, qa);
  const double r = boundary_r(a.q, a.q_ref, n_q_heads, a.first, grp, s_bpart);
  const bool fire = a.first || r < a.tau;
  if (c == 0 && kvh == 0 && tid == 0) {
    if (a.r_out) a.r_out[grp] = r;
    a.fire_out[grp] = (uint8_t)(fire ? 1 : 0);
  }
  if (c == 0 && w == 0)
    store_slice(a.k_new, a.v_new, a.k_local, a.v_local, a.window, a.step, a.seg_len, a.evict_seg, a.reps,
                a.unit_start, a.unit_size, a.units_cap, a.n_clusters, a.k_pool, a.v_pool, a.pool_rows, a.prompt_len,
                s, lane);

  // attention LDS (after the selection's, which it may reuse)
  float4 (*s_p)[NM][64] = reinterpret_cast<float4 (*)[NM][64]>(smem);
  float (*s_m)[G] = reinterpret_cast<float (*)[G]>(s_p + NW);
  float (*s_l)[G] = s_m + NW;
  float (*s_acc)[G][kHeadDim] = reinterpret_cast<float (*)[G][kHeadDim]>(s_l + NW);
  float2* s_ml = reinterpret_cast<float2*>(s_acc + NW);
  int* s_rows = reinterpret_cast<int*>(s_ml + nb * G);
  auto clamp_row = [&](int row) { return (int)min<int64_t>(max(row, 0), a.pool_rows - 1); };
  if (fire) {
    const bool selected = select_part<uint16_t, G, true>(
        a.q, a.n_kv_heads, s, c, nb, a.scale, a.reps, a.units_cap, a.n_units, a.n_pad, a.budget, a.unit_start,
        a.unit_size, a.sel_units, a.n_sel_units, a.n_sel, a.sel_rows, a.scores_out, a.logit_ws, a.part_max,
        a.sel_counter + s * kStepSyncStride, smem);
    if (selected) {
      // the list is out before the flag goes up
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      if (tid == 0) __hip_atomic_store(a.ready + s * kStepSyncStride, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
      if (tid == 0) {
        int polls = 0;
        while (__hip_atomic_load(a.ready + s * kStepSyncStride, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) {
          if (++polls >= a.spin_limit) {
            __hip_atomic_store(a.status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            break;
          }
          __builtin_amdgcn_s_sleep(8);
        }
      }
      __syncthreads();
    }
    nsel = __hip_atomic_load(a.n_sel + s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    for (int i = tid; p0 + i < sel_hi; i += kSelThreads)
      s_rows[i] = clamp_row(__hip_atomic_load(rl + p0 + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    load_attn_q<G>(a.q + (size_t)s * G * kHeadDim, lane, qa);   // not kept in registers across the selection
  } else {
#pragma unroll
    for (int e = 0; e < kStepListEarly; ++e) {
      const int i = tid + e * kSelThreads;
      if (p0 + i < sel_hi) s_rows[i] = clamp_row(early[e]);
    }
    for (int i = tid + kStepListEarly * kSelThreads; p0 + i < sel_hi; i += kSelThreads)
      s_rows[i] = clamp_row(__hip_atomic_load(rl + p0 + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
  }
  __syncthreads();
  nsel = max(0, min(nsel, a.budget));

  // the chunk's rows: 16-row tiles t = w, w + NW, ...
  const uint16_t* kb = a.k_pool + (size_t)s * a.pool_rows * kHeadDim;
  const uint16_t* vb = a.v_pool + (size_t)s * a.pool_rows * kHeadDim;
  const uint16_t* kl = a.k_local + (size_t)s * a.window * kHeadDim;
  const uint16_t* vl = a.v_local + (size_t)s * a.window * kHeadDim;
  const uint16_t* kn = a.k_new + (size_t)s * kHeadDim;
  const uint16_t* vn = a.v_new + (size_t)s * kHeadDim;
  const int newest = a.step % a.window;
  // the row at position pos of the chunk, or NULL if there is none
  auto row_ptr = [&](int pos, const uint16_t* pool, const uint16_t* ring, const uint16_t* cur) -> const uint16_t* {
    if (pos >= p1) return nullptr;
    if (pos < a.budget) return pos < nsel ? pool + (size_t)s_rows[pos - p0] * kHeadDim : nullptr;
    int slot = a.local_start + (pos - a.budget);   // local_start < window and pos - budget < n_local <= window
    slot -= slot >= a.window ? a.window : 0;
    return slot == newest ? cur : ring + (size_t)slot * kHeadDim;
  };
  auto load_tile = [&](int t, uint4 (&kx)[4], uint4 (&vx)[4]) -> bool {
    const int tb = p0 + 16 * t;
    const uint16_t* kp = row_ptr(tb + p16, kb, kl, kn);
#pragma unroll
    for (int cc = 0; cc < 4; ++cc) kx[cc] = kp ? *reinterpret_cast<const uint4*>(kp + 32 * cc + 8 * g) : uint4{};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint16_t* vp = row_ptr(tb + 4 * k + g, vb, vl, vn);
      vx[k] = vp ? *reinterpret_cast<const uint4*>(vp + 8 * p16) : uint4{};
    }
    return kp != nullptr;
  };
  // the block has read q_ref: count it in at the group's counter, after its
  // main loads (a wave's loads complete in order, and this atomic, on one
  // address for the whole group, returns late)
  int grp_old = 0;
  bool arrived = false;
  auto arrive_group = [&]() {
    if (arrived) return;
    arrived = true;
    __builtin_amdgcn_sched_barrier(0);
    if (tid == 0)
      grp_old = __hip_atomic_fetch_add(a.grp_counter + grp * kStepSyncStride, 1, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
  };
  float m[G], l[G], acc[G][8];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    m[j] = -__builtin_inff();
    l[j] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[j][e] = 0.f;
  }
  const float qscale = (float)a.scale * kLog2e;
  const int n_tiles = (p1 - p0 + 15) / 16;
  constexpr int kInFlight = G == 8 ? 1 : 2;   // tiles per wave in flight (G = 8: registers for one)
  for (int t = w; t < n_tiles; t += kInFlight * NW) {
    uint4 kx0[4], vx0[4], kx1[4], vx1[4];
    const bool two = kInFlight == 2 && t + NW < n_tiles;
    const bool kv0 = load_tile(t, kx0, vx0);
    const bool kv1 = two ? load_tile(t + NW, kx1, vx1) : false;
    arrive_group();
    attn_mfma_tile<G>(qa, kx0, vx0, kv0, qscale, m, l, acc, s_p[w], lane);
    if (two) attn_mfma_tile<G>(qa, kx1, vx1, kv1, qscale, m, l, acc, s_p[w], lane);
  }
  arrive_group();
  attn_wave_to_lds<G>(m, l, acc, s_m[w], s_l[w], s_acc[w], lane);
  __syncthreads();
  const bool done = attn_block_merge<G, NW, true>(s_m, s_l, s_acc, tid, s, c, nb, a.part, a.out, a.out_bf16,
                                                  a.lse_out, a.attn_counter + s * kStepSyncStride, s_ml);
  if (done && fire && tid == 0)
    __hip_atomic_store(a.ready + s * kStepSyncStride, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

  // the group's last block to arrive moves its reference query
  if (tid == 0) s_grp_last = grp_old == a.n_kv_heads * nb - 1;
  __syncthreads();
  if (!s_grp_last) return;
  if (tid == 0) __hip_atomic_store(a.grp_counter + grp * kStepSyncStride, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (a.mode == LOUISKV_REF_PREV || fire) {
    const size_t base = (size_t)grp * n_q_heads * kHeadDim;
    for (int i = tid; i < n_q_heads * kHeadDim / 8; i += kSelThreads)
      reinterpret_cast<uint4*>(a.q_ref + base)[i] = reinterpret_cast<const uint4*>(a.q + base)[i];
  }
}

// One wave per (slice, head): merge the chunk partials.
template <class TO>
__global__ __launch_bounds__(256)
void attn_combine_kernel(const float* __restrict__ part, int n_chunks, int G, int64_t n_rows,
                         TO* __restrict__ out, float* __restrict__ lse_out) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n_rows) return;
  const int lane = threadIdx.x & 63;
  const int64_t s = row / G;
  const int j = (int)(row - s * G);
  const size_t pstride = 2 + kHeadDim;
  const float* p = part + (size_t)s * n_chunks * G * pstride + (size_t)j * pstride;
  float mm = -__builtin_inff();
  for (int c = 0; c < n_chunks; ++c) mm = fmaxf(mm, p[(size_t)c * G * pstride]);
  float ll = 0.f, a0 = 0.f, a1 = 0.f;
  if (mm != -__builtin_inff()) {
    for (int c = 0; c < n_chunks; ++c) {
      const float* pc = p + (size_t)c * G * pstride;
      const float w = __builtin_amdgcn_exp2f(pc[0] - mm);
      ll += pc[1] * w;
      a0 += pc[2 + 2 * lane] * w;
      a1 += pc[2 + 2 * lane + 1] * w;
    }
  }
  const float inv = ll > 0.f ? 1.f / ll : 0.f;
  TO* o = out + (size_t)row * kHeadDim;
  store_from_f32(o, 2 * lane, a0 * inv);
  store_from_f32(o, 2 * lane + 1, a1 * inv);
  // partial maxima are in base 2: lse = ln 2 * (m + log2 l)
  if (lse_out && lane == 0) lse_out[row] = ll > 0.f ? 0.6931471805599453f * (mm + log2f(ll)) : -__builtin_inff();
}

int check_dtype(int dtype) {
  if (dtype != LOUISKV_F32 && dtype != LOUISKV_BF16) return fail(LOUISKV_ERR_DTYPE, "unknown dtype %d", dtype);
  return LOUISKV_OK;
}

size_t retrieve_ws_bytes(int64_t S, int units_cap, int budget) {
  Carver cv(nullptr);
  cv.take<double>(logit_ws_doubles(S, units_cap));
  cv.take<int32_t>((size_t)S * std::max(budget, 1));
  return align_up(cv.used, 256);
}

constexpr int kAttnMaxListRows = 8192;   // row-list entries one block stages in LDS (32 KB)

int attn_chunks(int64_t S, int buf_rows, int window, bool indexed) {
  const int64_t cap = (int64_t)buf_rows + window;
  const int64_t by_rows = std::max<int64_t>(1, (cap + kAttnMinRows - 1) / kAttnMinRows);
  const int64_t by_grid = std::max<int64_t>(1, (kAttnTargetBlocks + S - 1) / S);
  int64_t nc = std::min(by_rows, by_grid);
  if (indexed) nc = std::max<int64_t>(nc, (cap + kAttnMaxListRows - 1) / kAttnMaxListRows);
  return (int)nc;
}

size_t attn_ws_bytes(int64_t S, int G, int buf_rows, int window, bool indexed) {
  const int nc = attn_chunks(S, buf_rows, window, indexed);
  return nc == 1 ? 0 : align_up((size_t)S * nc * G * (2 + kHeadDim) * sizeof(float), 256);
}

// Chunks per slice of the fused decode step's bf16 attention: kStepAttnRows
// rows each, whatever the slice count (the step serves few slices at a time).
int step_attn_chunks(int buf_rows, int window) {
  return std::max(1, (int)(((int64_t)buf_rows + window + kStepAttnRows - 1) / kStepAttnRows));
}

// Partials of the fused step's attention (merged in-kernel), by dtype (bf16:
// the two-launch step's chunks or the one-launch step's blocks per slice).
size_t step_attn_part_bytes(int64_t S, int G, int buf_rows, int window, int dtype) {
  const int nc = dtype == LOUISKV_BF16 ? std::max(step_attn_chunks(buf_rows, window), kStepMaxBlocks)
                                       : attn_chunks(S, buf_rows, window, true);
  return nc == 1 ? 0 : align_up((size_t)S * nc * G * (2 + kHeadDim) * sizeof(float), 256);
}

}  // namespace
}  // namespace louiskv

using namespace louiskv;

extern "C" int louiskv_boundary_check(const void* q, void* q_ref, int32_t dtype, int64_t n_groups, int32_t n_q_heads,
                                      int32_t d, double tau, int32_t mode, int32_t first_step, double* r_out,
                                      uint8_t* fire_out, void* stream) {
  if (!q || !q_ref || !fire_out) return fail(LOUISKV_ERR_NULL, "q, q_ref and fire_out are required");
  int st = check_dtype(dtype);
  if (st) return st;
  if (d != kHeadDim) return fail(LOUISKV_ERR_UNSUPPORTED, "head dim %d not supported (only 128)", d);
  if (n_groups < 1 || n_q_heads < 1 || n_groups > INT32_MAX)
    return fail(LOUISKV_ERR_SHAPE, "n_groups=%lld n_q_heads=%d", (long long)n_groups, n_q_heads);
  if (mode != LOUISKV_REF_PREV && mode != LOUISKV_REF_ANCHOR) return fail(LOUISKV_ERR_SHAPE, "unknown mode %d", mode);
  hipStream_t s = as_stream(stream);
  if (dtype == LOUISKV_BF16)
    boundary_kernel<uint16_t><<<(unsigned)n_groups, 256, 0, s>>>(static_cast<const uint16_t*>(q),
                                                                 static_cast<uint16_t*>(q_ref), n_q_heads, tau, mode,
                                                                 first_step ? 1 : 0, r_out, fire_out);
  else
    boundary_kernel<float><<<(unsigned)n_groups, 256, 0, s>>>(static_cast<const float*>(q), static_cast<float*>(q_ref),
                                                              n_q_heads, tau, mode, first_step ? 1 : 0, r_out,
                                                              fire_out);
  LKV_CHECK_LAUNCH();
  return LOUISKV_OK;
}

namespace louiskv {
namespace {
// Fixed-stride trigger: every group fires on the steps that are multiples of
// the stride.
__global__ void fire_every_kernel(uint8_t* __restrict__ fire, int64_t n_groups, uint8_t value) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g < n_groups) fire[g] = value;
}
}  // namespace
}  // namespace louiskv

extern "C" int louiskv_fire_every(uint8_t* fire_out, int64_t n_groups, int32_t step, int32_t stride, void* stream) {
  if (!fire_out) return fail(LOUISKV_ERR_NULL, "fire_out is required");
  if (n_groups < 1 || n_groups > INT32_MAX || step < 0 || stride < 1)
    return fail(LOUISKV_ERR_SHAPE, "n_groups=%lld step=%d stride=%d", (long long)n_groups, step, stride);
  fire_every_kernel<<<(unsigned)((n_groups + 255) / 256), 256, 0, as_stream(stream)>>>(
      fire_out, n_groups, (uint8_t)(step % stride == 0 ? 1 : 0));
  LKV_CHECK_LAUNCH();
  return LOUISKV_OK;
}

extern "C" int louiskv_segment_output(const void* k_new, const void* v_new, int32_t dtype, int64_t n_slices, int32_t d,
                                      void* k_local, void* v_local, int32_t window, int32_t step, int32_t seg_len,
                                      float* reps, int32_t* unit_start, int32_t* unit_size, int32_t units_cap,
                                      int32_t n_clusters, void* k_pool, void* v_pool, int64_t pool_rows,
                                      int32_t prompt_len, int32_t pool_on_host, void* stream) {
  if (!k_new || !v_new || !k_local || !v_local) return fail(LOUISKV_ERR_NULL, "k_new, v_new, k_local, v_local required");
  int st = check_dtype(dtype);
  if (st) return st;
  if (pool_on_host && ((st = device_view_of_host_pool(k_pool, &k_pool)) || (st = device_view_of_host_pool(v_pool, &v_pool))))
    return st;
  if (d != kHeadDim) return fail(LOUISKV_ERR_UNSUPPORTED, "head dim %d not supported (only 128)", d);
  if (n_slices < 1 || n_slices > INT32_MAX) return fail(LOUISKV_ERR_SHAPE, "n_slices=%lld", (long long)n_slices);
  int32_t ev = -1, n_ev = 0;
  st = louiskv_window_info(step, window, seg_len, &ev, &n_ev, nullptr, nullptr);
  if (st) return st;
  if (ev >= 0) {
    if (!reps || !unit_start || !unit_size) return fail(LOUISKV_ERR_NULL, "unit tables required for an eviction");
    if (n_clusters < 0 || (int64_t)n_clusters + ev >= units_cap)
      return fail(LOUISKV_ERR_SHAPE, "unit %d exceeds units_cap=%d", n_clusters + ev, units_cap);
    if ((k_pool || v_pool) && (int64_t)prompt_len + (int64_t)(ev + 1) * seg_len > pool_rows)
      return fail(LOUISKV_ERR_SHAPE, "segment rows exceed pool_rows=%lld", (long long)pool_rows);
    if (v_pool && !k_pool) return fail(LOUISKV_ERR_NULL, "v_pool given without k_pool");
  }
  hipStream_t s = as_stream(stream);
  if (dtype == LOUISKV_BF16)
    store_decode_kernel<uint16_t><<<(unsigned)n_slices, 64, 0, s>>>(
        static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new), static_cast<uint16_t*>(k_local),
        static_cast<uint16_t*>(v_local), window, step, seg_len, ev, reps, unit_start, unit_size, units_cap, n_clusters,
        static_cast<uint16_t*>(k_pool), static_cast<uint16_t*>(v_pool), pool_rows, prompt_len);
  else
    store_decode_kernel<float><<<(unsigned)n_slices, 64, 0, s>>>(
        static_cast<const float*>(k_new), static_cast<const float*>(v_new), static_cast<float*>(k_local),
        static_cast<float*>(v_local), window, step, seg_len, ev, reps, unit_start, unit_size, units_cap, n_clusters,
        static_cast<float*>(k_pool), static_cast<float*>(v_pool), pool_rows, prompt_len);
  LKV_CHECK_LAUNCH();
  return LOUISKV_OK;
}

extern "C" int louiskv_decode_prologue(const void* q, void* q_ref, int32_t dtype, int64_t n_groups,
                                       int32_t n_q_heads, int32_t d, double tau, int32_t mode, int32_t first_step,
                                       double* r_out, uint8_t* fire_out, const void* k_new, const void* v_new,
                                       int64_t n_slices, void* k_local, void* v_local, int32_t window, int32_t step,
                                       int32_t seg_len, float* reps, int32_t* unit_start, int32_t* unit_size,
                                       int32_t units_cap, int32_t n_clusters, void* k_pool, void* v_pool,
                                       int64_t pool_rows, int32_t prompt_len, int32_t pool_on_host, void* stream) {
  if (!q || !q_ref || !fire_out) return fail(LOUISKV_ERR_NULL, "q, q_ref and fire_out are required");
  if (!k_new || !v_new || !k_local || !v_local) return fail(LOUISKV_ERR_NULL, "k_new, v_new, k_local, v_local required");
  int st = check_dtype(dtype);
  if (st) return st;
  if (d != kHeadDim) return fail(LOUISKV_ERR_UNSUPPORTED, "head dim %d not supported (only 128)", d);
  if (n_groups < 1 || n_q_heads < 1 || n_slices < 1 || (n_slices + 3) / 4 + n_groups > INT32_MAX)
    return fail(LOUISKV_ERR_SHAPE, "n_groups=%lld n_q_heads=%d n_slices=%lld", (long long)n_groups, n_q_heads,
                (long long)n_slices);
  if (mode != LOUISKV_REF_PREV && mode != LOUISKV_REF_ANCHOR) return fail(LOUISKV_ERR_SHAPE, "unknown mode %d", mode);
  if (pool_on_host && ((st = device_view_of_host_pool(k_pool, &k_pool)) || (st = device_view_of_host_pool(v_pool, &v_pool))))
    return st;
  int32_t ev = -1, n_ev = 0;
  if ((st = louiskv_window_info(step, window, seg_len, &ev, &n_ev, nullptr, nullptr))) return st;
  if (ev >= 0) {
    if (!reps || !unit_start || !unit_size) return fail(LOUISKV_ERR_NULL, "unit tables required for an eviction");
    if (n_clusters < 0 || (int64_t)n_clusters + ev >= units_cap)
      return fail(LOUISKV_ERR_SHAPE, "unit %d exceeds units_cap=%d", n_clusters + ev, units_cap);
    if ((k_pool || v_pool) && (int64_t)prompt_len + (int64_t)(ev + 1) * seg_len > pool_rows)
      return fail(LOUISKV_ERR_SHAPE, "segment rows exceed pool_rows=%lld", (long long)pool_rows);
    if (v_pool && !k_pool) return fail(LOUISKV_ERR_NULL, "v_pool given without k_pool");
  }
  hipStream_t s = as_stream(stream);
  const unsigned grid = (unsigned)(n_groups + (n_slices + 3) / 4);
  if (dtype == LOUISKV_BF16)
    decode_prologue_kernel<uint16_t><<<grid, 256, 0, s>>>(
        static_cast<const uint16_t*>(q), static_cast<uint16_t*>(q_ref), n_q_heads, tau, mode, first_step ? 1 : 0,
        r_out, fire_out, (int)n_groups, static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new),
        static_cast<uint16_t*>(k_local), static_cast<uint16_t*>(v_local), n_slices, window, step, seg_len, ev, reps,
        unit_start, unit_size, units_cap, n_clusters, static_cast<uint16_t*>(k_pool), static_cast<uint16_t*>(v_pool),
        pool_rows, prompt_len);
  else
    decode_prologue_kernel<float><<<grid, 256, 0, s>>>(
        static_cast<const float*>(q), static_cast<float*>(q_ref), n_q_heads, tau, mode, first_step ? 1 : 0, r_out,
        fire_out, (int)n_groups, static_cast<const float*>(k_new), static_cast<const float*>(v_new),
        static_cast<float*>(k_local), static_cast<float*>(v_local), n_slices, window, step, seg_len, ev, reps,
        unit_start, unit_size, units_cap, n_clusters, static_cast<float*>(k_pool), static_cast<float*>(v_pool),
        pool_rows, prompt_len);
  LKV_CHECK_LAUNCH();
  return LOUISKV_OK;
}

extern "C" size_t louiskv_segment_state_ints(int32_t window) {
  return window >= 2 ? (size_t)(kSegRing + window) : 0;
}

extern "C" int louiskv_segment_state_init(int32_t* seg_state, int64_t n_slices, int32_t window, int32_t n_clusters,
                                          void* stream) {
  if (!seg_state) return fail(LOUISKV_ERR_NULL, "seg_state is required");
  if (window < 2 || n_slices < 1 || n_clusters < 1)
    return fail(LOUISKV_ERR_SHAPE, "window=%d n_slices=%lld n_clusters=%d", window, (long long)n_slices, n_clusters);
  const int stride = kSegRing + window;
  const int64_t n = n_slices * stride;
  seg_state_init_kernel<<<(unsigned)((n + 255) / 256), 256, 0, as_stream(stream)>>>(seg_state, n_slices, stride,
                                                                                   n_clusters);
  LKV_CHECK_LAUNCH();
  return LOUISKV_OK;
}

extern "C" int louiskv_segment_output_boundary(const void* k_new, const void* v_new, int32_t dtype, int64_t n_slices,
                                               int32_t n_kv_heads, int32_t d, void* k_local, void* v_local,
                                               int32_t window, int32_t step, int32_t seg_max, const uint8_t* fire,
                                               int32_t* seg_state, float* reps, int32_t* unit_start,
                                               int32_t* unit_size, int32_t units_cap, int32_t n_clusters,
                                               void* k_pool, void* v_pool, int64_t pool_rows, int32_t prompt_len,
                                               int32_t pool_on_host, void* stream) {
  if (!k_new || !v_new || !k_local || !v_local || !seg_state)
    return fail(LOUISKV_ERR_NULL, "k_new, v_new, k_local, v_local and seg_state are required");
  if (!reps || !unit_start || !unit_size) return fail(LOUISKV_ERR_NULL, "unit tables are required");
  if (v_pool && !k_pool) return fail(LOUISKV_ERR_NULL, "v_pool given without k_pool");
  int st = check_dtype(dtype);
  if (st) return st;
  if (pool_on_host && ((st = device_view_of_host_pool(k_pool, &k_pool)) || (st = device_view_of_host_pool(v_pool, &v_pool))))
    return st;
  if (d != kHeadDim) return fail(LOUISKV_ERR_UNSUPPORTED, "head dim %d not supported (only 128)", d);
  if (n_kv_heads < 1 || n_slices < 1 || n_slices % n_kv_heads != 0 || n_slices > INT32_MAX)
    return fail(LOUISKV_ERR_SHAPE, "n_slices=%lld must be a positive multiple of n_kv_heads=%d", (long long)n_slices,
                n_kv_heads);
  if (window < 2 || seg_max < 1 || seg_max >= window)
    return fail(LOUISKV_ERR_SHAPE, "need 1 <= seg_max=%d < window=%d", seg_max, window);
  if (step < 0) return fail(LOUISKV_ERR_SHAPE, "step=%d < 0", step);
  if (n_clusters < 1 || n_clusters > units_cap)
    return fail(LOUISKV_ERR_SHAPE, "n_clusters=%d must be in [1, units_cap=%d]", n_clusters, units_cap);
  if (prompt_len < 0 || ((k_pool || v_pool) && pool_rows < prompt_len))
    return fail(LOUISKV_ERR_SHAPE, "prompt_len=%d pool_rows=%lld", prompt_len, (long long)pool_rows);
  hipStream_t s = as_stream(stream);
  if (dtype == LOUISKV_BF16)
    store_segmented_kernel<uint16_t><<<(unsigned)n_slices, 64, 0, s>>>(
        static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new), static_cast<uint16_t*>(k_local),
        static_cast<uint16_t*>(v_local), window, step, seg_max, fire, n_kv_heads, seg_state, reps, unit_start,
        unit_size, units_cap, n_clusters, static_cast<uint16_t*>(k_pool), static_cast<uint16_t*>(v_pool), pool_rows,
        prompt_len);
  else
    store_segmented_kernel<float><<<(unsigned)n_slices, 64, 0, s>>>(
        static_cast<const float*>(k_new), static_cast<const float*>(v_new), static_cast<float*>(k_local),
        static_cast<float*>(v_local), window, step, seg_max, fire, n_kv_heads, seg_state, reps, unit_start, unit_size,
        units_cap, n_clusters, static_cast<float*>(k_pool), static_cast<float*>(v_pool), pool_rows, prompt_len);
  LKV_CHECK_LAUNCH();
  return LOUISKV_OK;
}

extern "C" size_t louiskv_retrieve_workspace_size(int64_t n_slices, int32_t units_cap, int32_t budget) {
  if (n_slices < 1 || units_cap < 1 || budget < 0) return 0;
  return retrieve_ws_bytes(n_slices, units_cap, budget);
}

namespace louiskv {
namespace {

// Arguments shared by both retrieval entry points, then the scoring/selection
// kernel, whose pool-row list goes to `rows` ([n_slices][budget]).
int score_and_select(const void* q, int32_t dtype, int64_t n_slices, int32_t n_kv_heads, int32_t group_size, int32_t d,
                     double scale, const float* reps, const int32_t* unit_start, const int32_t* unit_size,
                     int32_t units_cap, int32_t n_units, int32_t budget, const uint8_t* fire, int32_t* sel_units,
                     int32_t* n_sel_units, int32_t* n_sel, int32_t* rows, double* scores_out, double* logit_ws,
                     const int32_t* seg_state, int32_t seg_stride, hipStream_t s, int32_t slice_div = 1) {
  if (n_units < 1 || n_units > units_cap || n_units > kMaxUnits)
    return fail(LOUISKV_ERR_SHAPE, "n_units=%d must be in [1, min(units_cap=%d, %d)]", n_units, units_cap, kMaxUnits);
  int n_pad = 64;                     // whole 64-key chunks for the in-wave sort steps
  while (n_pad < n_units) n_pad <<= 1;
  const size_t lds = (size_t)n_pad * (sizeof(uint64_t) + 2 * sizeof(int));
  (void)d;
  const int parts = logit_parts(n_slices, n_units);
  if ((int64_t)n_slices * parts > INT32_MAX) return fail(LOUISKV_ERR_SHAPE, "problem too large for one launch");
  int st = LOUISKV_OK;
  // More slices than compute units: 256-thread blocks, two to a compute unit,
  // so that one block's selection overlaps the other's logit loads (the
  // scores are the same for both block sizes); else one 512-thread block each.
  const bool small_blocks = n_slices > device_cu_count();
#define LKV_SEL_NT(T, G, NT)                                                                                           \
  if ((st = check_lds(reinterpret_cast<const void*>(&score_select_kernel<T, G, NT>), lds))) return st;                 \
  score_select_kernel<T, G, NT><<<(unsigned)n_slices, NT, lds, s>>>(                                                   \
      static_cast<const T*>(q), n_kv_heads, scale, reps, unit_start, unit_size, units_cap, n_units, budget, fire,    \
      sel_units, n_sel_units, n_sel, scores_out, logit_ws, rows, n_pad, seg_state, seg_stride, slice_div,            \
      parts == 1 ? 1 : 0)
#define LKV_SEL(T, G)                                                                                                  \
  if (parts > 1)                                                                                                       \
    unit_logits_kernel<T, G><<<(unsigned)(n_slices * parts), kLogitThreads, 0, s>>>(                                   \
        static_cast<const T*>(q), n_kv_heads, scale, reps, units_cap, n_units, fire, logit_ws, seg_state,            \
        seg_stride, slice_div, parts);                                                                                \
  if (small_blocks) {                                                                                                  \
    LKV_SEL_NT(T, G, kSmallSelThreads);                                                                                \
  } else {                                                                                                             \
    LKV_SEL_NT(T, G, kSelThreads);                                                                                     \
  }
#define LKV_SEL_G(T)                  \
  switch (group_size) {               \
    case 1: LKV_SEL(T, 1); break;     \
    case 2: LKV_SEL(T, 2); break;     \
    case 3: LKV_SEL(T, 3); break;     \
    case 4: LKV_SEL(T, 4); break;     \
    case 5: LKV_SEL(T, 5); break;     \
    case 6: LKV_SEL(T, 6); break;     \
    case 7: LKV_SEL(T, 7); break;     \
    default: LKV_SEL(T, 8); break;    \
  }
  if (dtype == LOUISKV_BF16) {
    LKV_SEL_G(uint16_t)
  } else {
    LKV_SEL_G(float)
  }
#undef LKV_SEL_G
#undef LKV_SEL
#undef LKV_SEL_NT
  LKV_CHECK_LAUNCH();
  return LOUISKV_OK;
}

int check_retrieve_common(const void* q, int32_t dtype, int64_t n_slices, int32_t n_kv_heads, int32_t group_size,
                          int32_t d, const float* reps, const int32_t* unit_start, const int32_t* unit_size,
                          int32_t units_cap, int32_t n_units, int32_t budget, const int32_t* sel_units,
                          const int32_t* n_sel_units, const int32_t* n_sel) {
  if (!q || !reps || !unit_start || !unit_size || !sel_units || !n_sel_units || !n_sel)
    return fail(LOUISKV_ERR_NULL, "q, reps, unit tables and selection outputs are required");
  int st = check_dtype(dtype);
  if (st) return st;
  if (d != kHeadDim) return fail(LOUISKV_ERR_UNSUPPORTED, "head dim %d not supported (only 128)", d);
  if (n_kv_heads < 1 || n_slices < 1 || n_slices % n_kv_heads != 0 || n_slices > INT32_MAX)
    return fail(LOUISKV_ERR_SHAPE, "n_slices=%lld must be a positive multiple of n_kv_heads=%d", (long long)n_slices,
                n_kv_heads);
  if (group_size < 1 || group_size > kMaxGroupSize)
    return fail(LOUISKV_ERR_UNSUPPORTED, "group_size=%d must be in [1, %d]", group_size, kMaxGroupSize);
  if (n_units < 1 || n_units > units_cap || n_units > kMaxUnits)
    return fail(LOUISKV_ERR_SHAPE, "n_units=%d must be in [1, min(units_cap=%d, %d)]", n_units, units_cap, kMaxUnits);
  if (budget < 0) return fail(LOUISKV_ERR_SHAPE, "budget=%d < 0", budget);
  return LOUISKV_OK;
}

}  // namespace
}  // namespace louiskv

namespace louiskv {
namespace {
int retrieve_gather(const void* q, int32_t dtype, int64_t n_slices, int32_t n_kv_heads, int32_t group_size, int32_t d,
                    double scale, const float* reps, const int32_t* unit_start, const int32_t* unit_size,
                    int32_t units_cap, int32_t n_units, const void* k_pool, const void* v_pool, int64_t pool_rows,
                    int32_t pool_on_host, int32_t budget, const uint8_t* fire, int32_t* sel_units,
                    int32_t* n_sel_units, int32_t* n_sel, void* k_buf, void* v_buf, double* scores_out,
                    void* workspace, size_t workspace_bytes, const int32_t* seg_state, int32_t seg_stride,
                    void* stream) {
  int st = check_retrieve_common(q, dtype, n_slices, n_kv_heads, group_size, d, reps, unit_start, unit_size, units_cap,
                                 n_units, budget, sel_units, n_sel_units, n_sel);
  if (st) return st;
  if (!k_pool || !v_pool || !k_buf || !v_buf) return fail(LOUISKV_ERR_NULL, "k_pool, v_pool, k_buf, v_buf required");
  void* kpd = const_cast<void*>(k_pool);
  void* vpd = const_cast<void*>(v_pool);
  if (pool_on_host && ((st = device_view_of_host_pool(k_pool, &kpd)) || (st = device_view_of_host_pool(v_pool, &vpd))))
    return st;
  const size_t need = retrieve_ws_bytes(n_slices, units_cap, budget);
  if (!workspace || workspace_bytes < need)
    return fail(LOUISKV_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, workspace_bytes);
  Carver cv(workspace);
  double* logit_ws = cv.take<double>(logit_ws_doubles(n_slices, units_cap));
  int32_t* row_ws = cv.take<int32_t>((size_t)n_slices * std::max(budget, 1));
  hipStream_t s = as_stream(stream);
  if ((st = score_and_select(q, dtype, n_slices, n_kv_heads, group_size, d, scale, reps, unit_start, unit_size,
                             units_cap, n_units, budget, fire, sel_units, n_sel_units, n_sel, row_ws, scores_out,
                             logit_ws, seg_state, seg_stride, s)))
    return st;
  if (budget > 0) {
    const int rpb = 128;
    const int bps = (budget + rpb - 1) / rpb;
    const unsigned grid = (unsigned)(n_slices * bps);
    if (dtype == LOUISKV_BF16)
      gather_kernel<uint16_t><<<grid, 256, 0, s>>>(static_cast<const uint16_t*>(kpd),
                                                   static_cast<const uint16_t*>(vpd), pool_rows, row_ws, n_sel, fire,
                                                   n_kv_heads, budget, bps, rpb, static_cast<uint16_t*>(k_buf),
                                                   static_cast<uint16_t*>(v_buf));
    else
      gather_kernel<float><<<grid, 256, 0, s>>>(static_cast<const float*>(kpd), static_cast<const float*>(vpd),
                                                pool_rows, row_ws, n_sel, fire, n_kv_heads, budget, bps, rpb,
                                                static_cast<float*>(k_buf), static_cast<float*>(v_buf));
    LKV_CHECK_LAUNCH();
  }
  return LOUISKV_OK;
}

int retrieve_rows(const void* q, int32_t dtype, int64_t n_slices, int32_t n_kv_heads, int32_t group_size, int32_t d,
                  double scale, const float* reps, const int32_t* unit_start, const int32_t* unit_size,
                  int32_t units_cap, int32_t n_units, int32_t budget, const uint8_t* fire, int32_t* sel_units,
                  int32_t* n_sel_units, int32_t* n_sel, int32_t* sel_rows, double* scores_out, void* workspace,
                  size_t workspace_bytes, const int32_t* seg_state, int32_t seg_stride, void* stream) {
  int st = check_retrieve_common(q, dtype, n_slices, n_kv_heads, group_size, d, reps, unit_start, unit_size, units_cap,
                                 n_units, budget, sel_units, n_sel_units, n_sel);
  if (st) return st;
  if (budget > 0 && !sel_rows) return fail(LOUISKV_ERR_NULL, "sel_rows is required when budget > 0");
  const size_t need = align_up(logit_ws_doubles(n_slices, units_cap) * sizeof(double), 256);
  if (!workspace || workspace_bytes < need)
    return fail(LOUISKV_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, workspace_bytes);
  return score_and_select(q, dtype, n_slices, n_kv_heads, group_size, d, scale, reps, unit_start, unit_size, units_cap,
                          n_units, budget, fire, sel_units, n_sel_units, n_sel, sel_rows, scores_out,
                          static_cast<double*>(workspace), seg_state, seg_stride, as_stream(stream));
}

int check_seg_state(const int32_t* seg_state, int32_t window) {
  if (!seg_state) return fail(LOUISKV_ERR_NULL, "seg_state is required");
  if (window < 2) return fail(LOUISKV_ERR_SHAPE, "window=%d must be >= 2", window);
  return LOUISKV_OK;
}
}  // namespace
}  // namespace louiskv

extern "C" int louiskv_retrieve(const void* q, int32_t dtype, int64_t n_slices, int32_t n_kv_heads, int32_t group_size,
                                int32_t d, double scale, const float* reps, const int32_t* unit_start,
                                const int32_t* unit_size, int32_t units_cap, int32_t n_units, const void* k_pool,
                                const void* v_pool, int64_t pool_rows, int32_t pool_on_host, int32_t budget,
                                const uint8_t* fire, int32_t* sel_units, int32_t* n_sel_units, int32_t* n_sel,
                                void* k_buf, void* v_buf, double* scores_out, void* workspace, size_t workspace_bytes,
                                void* stream) {
  return retrieve_gather(q, dtype, n_slices, n_kv_heads, group_size, d, scale, reps, unit_start, unit_size, units_cap,
                         n_units, k_pool, v_pool, pool_rows, pool_on_host, budget, fire, sel_units, n_sel_units, n_sel,
                         k_buf, v_buf, scores_out, workspace, workspace_bytes, nullptr, 0, stream);
}

extern "C" int louiskv_retrieve_seg(const void* q, int32_t dtype, int64_t n_slices, int32_t n_kv_heads,
                                    int32_t group_size, int32_t d, double scale, const float* reps,
                                    const int32_t* unit_start, const int32_t* unit_size, int32_t units_cap,
                                    int32_t max_units, const int32_t* seg_state, int32_t window, const void* k_pool,
                                    const void* v_pool, int64_t pool_rows, int32_t pool_on_host, int32_t budget,
                                    const uint8_t* fire, int32_t* sel_units, int32_t* n_sel_units, int32_t* n_sel,
                                    void* k_buf, void* v_buf, double* scores_out, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  int st = check_seg_state(seg_state, window);
  if (st) return st;
  return retrieve_gather(q, dtype, n_slices, n_kv_heads, group_size, d, scale, reps, unit_start, unit_size, units_cap,
                         max_units, k_pool, v_pool, pool_rows, pool_on_host, budget, fire, sel_units, n_sel_units,
                         n_sel, k_buf, v_buf, scores_out, workspace, workspace_bytes, seg_state, kSegRing + window,
                         stream);
}

extern "C" size_t louiskv_retrieve_rows_workspace_size(int64_t n_slices, int32_t units_cap) {
  if (n_slices < 1 || units_cap < 1) return 0;
  return align_up(logit_ws_doubles(n_slices, units_cap) * sizeof(double), 256);
}

extern "C" int louiskv_retrieve_rows(const void* q, int32_t dtype, int64_t n_slices, int32_t n_kv_heads,
                                     int32_t group_size, int32_t d, double scale, const float* reps,
                                     const int32_t* unit_start, const int32_t* unit_size, int32_t units_cap,
                                     int32_t n_units, int32_t budget, const uint8_t* fire, int32_t* sel_units,
                                     int32_t* n_sel_units, int32_t* n_sel, int32_t* sel_rows, double* scores_out,
                                     void* workspace, size_t workspace_bytes, void* stream) {
  return retrieve_rows(q, dtype, n_slices, n_kv_heads, group_size, d, scale, reps, unit_start, unit_size, units_cap,
                       n_units, budget, fire, sel_units, n_sel_units, n_sel, sel_rows, scores_out, workspace,
                       workspace_bytes, nullptr, 0, stream);
}

extern "C" int louiskv_retrieve_rows_seg(const void* q, int32_t dtype, int64_t n_slices, int32_t n_kv_heads,
                                         int32_t group_size, int32_t d, double scale, const float* reps,
                                         const int32_t* unit_start, const int32_t* unit_size, int32_t units_cap,
                                         int32_t max_units, const int32_t* seg_state, int32_t window, int32_t budget,
                                         const uint8_t* fire, int32_t* sel_units, int32_t* n_sel_units,
                                         int32_t* n_sel, int32_t* sel_rows, double* scores_out, void* workspace,
                                         size_t workspace_bytes, void* stream) {
  int st = check_seg_state(seg_state, window);
  if (st) return st;
  return retrieve_rows(q, dtype, n_slices, n_kv_heads, group_size, d, scale, reps, unit_start, unit_size, units_cap,
                       max_units, budget, fire, sel_units, n_sel_units, n_sel, sel_rows, scores_out, workspace,
                       workspace_bytes, seg_state, kSegRing + window, stream);
}

extern "C" size_t louiskv_sparse_decode_attn_workspace_size(int64_t n_slices, int32_t group_size, int32_t d,
                                                            int32_t buf_rows, int32_t window) {
  (void)d;
  if (n_slices < 1 || group_size < 1 || buf_rows < 0 || window < 0) return 0;
  return attn_ws_bytes(n_slices, group_size, buf_rows, window, false);
}

extern "C" size_t louiskv_sparse_decode_attn_rows_workspace_size(int64_t n_slices, int32_t group_size, int32_t d,
                                                                 int32_t budget, int32_t window) {
  (void)d;
  if (n_slices < 1 || group_size < 1 || budget < 0 || window < 0) return 0;
  return attn_ws_bytes(n_slices, group_size, budget, window, true);
}

namespace louiskv {
namespace {

struct AttnArgs {
  const void* q;
  int n_kv_heads;
  float scale;
  const void* k_src;
  const void* v_src;
  const int32_t* n_sel;
  int buf_rows;            // KV_critical rows per slice, or row-list entries per slice
  const int32_t* rows;     // row list, or NULL for the dense KV_critical
  int64_t src_rows;        // rows per slice of k_src/v_src
  const void* k_local;
  const void* v_local;
  int window, local_start, n_local, n_chunks;
  float* part;
  void* out;
  int out_bf16;
  float* lse_out;
  const int32_t* seg_state;   // per-slice windows (boundary-delimited segments) or NULL
  int seg_stride, n_tokens;
  unsigned grid;
  size_t lds;              // dynamic LDS for the staged row list
  int slice_div = 1;       // lists per KV-head slice (per-head selection: the group size)
  StepSync sync = {nullptr, nullptr, nullptr, 0};   // fused decode step: in-kernel merge, q_ref update
  int step_waves = 0;      // fused decode step, bf16: waves per block (0: the default block)
};

template <class T, int G, bool kIdx>
void launch_attn_partial(const AttnArgs& a, hipStream_t s) {
  attn_partial_kernel<T, G, kIdx><<<a.grid, attn_waves<T, G>() * 64, a.lds, s>>>(
      static_cast<const T*>(a.q), a.n_kv_heads, a.scale, static_cast<const T*>(a.k_src), static_cast<const T*>(a.v_src),
      a.n_sel, a.buf_rows, a.rows, a.src_rows, static_cast<const T*>(a.k_local), static_cast<const T*>(a.v_local),
      a.window, a.local_start, a.n_local, a.n_chunks, a.part, a.out, a.out_bf16, a.lse_out, a.seg_state,
      a.seg_stride, a.n_tokens, a.slice_div, a.sync);
}

template <int G, bool kIdx, int NW>
void launch_attn_mfma_nw(const AttnArgs& a, hipStream_t s) {
  attn_mfma_kernel<G, kIdx, NW><<<a.grid, NW * 64, a.lds, s>>>(
      static_cast<const uint16_t*>(a.q), a.n_kv_heads, a.scale, static_cast<const uint16_t*>(a.k_src),
      static_cast<const uint16_t*>(a.v_src), a.n_sel, a.buf_rows, a.rows, a.src_rows,
      static_cast<const uint16_t*>(a.k_local), static_cast<const uint16_t*>(a.v_local), a.window, a.local_start,
      a.n_local, a.n_chunks, a.part, a.out, a.out_bf16, a.lse_out, a.seg_state, a.seg_stride, a.n_tokens,
      a.slice_div, a.sync);
}

template <int G, bool kIdx>
void launch_attn_mfma(const AttnArgs& a, hipStream_t s) {
  if (kIdx && a.step_waves == kStepAttnWaves)
    launch_attn_mfma_nw<G, kIdx, kStepAttnWaves>(a, s);
  else
    launch_attn_mfma_nw<G, kIdx, attn_mfma_waves<G>()>(a, s);
}

template <bool kIdx>
void launch_attn(int dtype, int group_size, const AttnArgs& a, hipStream_t s) {
  if (dtype == LOUISKV_BF16) {
    switch (group_size) {
      case 1: launch_attn_mfma<1, kIdx>(a, s); break;
      case 2: launch_attn_mfma<2, kIdx>(a, s); break;
      case 4: launch_attn_mfma<4, kIdx>(a, s); break;
      default: launch_attn_mfma<8, kIdx>(a, s); break;
    }
  } else {
    switch (group_size) {
      case 1: launch_attn_partial<float, 1, kIdx>(a, s); break;
      case 2: launch_attn_partial<float, 2, kIdx>(a, s); break;
      case 4: launch_attn_partial<float, 4, kIdx>(a, s); break;
      default: launch_attn_partial<float, 8, kIdx>(a, s); break;
    }
  }
}

// Validation and launch shared by the dense (KV_critical) and the row-list
// entry points.
int sparse_decode_attn(const void* q, int32_t dtype, int64_t n_slices, int32_t n_kv_heads, int32_t group_size,
                       int32_t d, float scale, const void* k_src, const void* v_src, const int32_t* n_sel,
                       int32_t buf_rows, const int32_t* rows, int64_t src_rows, const void* k_local,
                       const void* v_local, int32_t window, int32_t local_start, int32_t n_local, void* out,
                       int32_t out_dtype, float* lse_out, void* workspace, size_t workspace_bytes, void* stream,
                       const int32_t* seg_state = nullptr, int32_t n_tokens = 0, int32_t slice_div = 1,
                       const StepSync* step_sync = nullptr) {
  const bool indexed = rows != nullptr;
  if (!q || !out || !n_sel) return fail(LOUISKV_ERR_NULL, "q, out and n_sel are required");
  if (buf_rows > 0 && (!k_src || !v_src))
    return fail(LOUISKV_ERR_NULL, indexed ? "k_pool/v_pool required when budget > 0"
                                          : "k_buf/v_buf required when buf_rows > 0");
  if (n_local > 0 && (!k_local || !v_local)) return fail(LOUISKV_ERR_NULL, "k_local/v_local required when n_local > 0");
  int st = check_dtype(dtype);
  if (st) return st;
  if ((st = check_dtype(out_dtype))) return st;
  if (d != kHeadDim) return fail(LOUISKV_ERR_UNSUPPORTED, "head dim %d not supported (only 128)", d);
  if (n_kv_heads < 1 || n_slices < 1 || n_slices % n_kv_heads != 0)
    return fail(LOUISKV_ERR_SHAPE, "n_slices=%lld must be a positive multiple of n_kv_heads=%d", (long long)n_slices,
                n_kv_heads);
  if (group_size != 1 && group_size != 2 && group_size != 4 && group_size != 8)
    return fail(LOUISKV_ERR_UNSUPPORTED, "group_size=%d must be 1, 2, 4 or 8", group_size);
  if (buf_rows < 0 || window < 0 || n_local < 0 || n_local > window || (window > 0 && (local_start < 0 || local_start >= window)))
    return fail(LOUISKV_ERR_SHAPE, "buf_rows=%d window=%d local_start=%d n_local=%d", buf_rows, window, local_start,
                n_local);
  if (indexed && buf_rows > 0 && src_rows < 1) return fail(LOUISKV_ERR_SHAPE, "pool_rows=%lld", (long long)src_rows);
  const bool step_bf16 = step_sync && indexed && dtype == LOUISKV_BF16;
  const int n_chunks = step_bf16 ? step_attn_chunks(buf_rows, window) : attn_chunks(n_slices, buf_rows, window, indexed);
  if ((int64_t)n_slices * n_chunks > INT32_MAX) return fail(LOUISKV_ERR_SHAPE, "problem too large for one launch");
  const size_t need = step_sync ? step_attn_part_bytes(n_slices, group_size, buf_rows, window, dtype)
                                : attn_ws_bytes(n_slices, group_size, buf_rows, window, indexed);
  if (need > 0 && (!workspace || workspace_bytes < need))
    return fail(LOUISKV_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, workspace_bytes);
  AttnArgs a;
  a.q = q; a.n_kv_heads = n_kv_heads; a.scale = scale; a.k_src = k_src; a.v_src = v_src; a.n_sel = n_sel;
  a.buf_rows = buf_rows; a.rows = rows; a.src_rows = indexed ? src_rows : buf_rows;
  a.k_local = k_local; a.v_local = v_local;
  a.window = window > 0 ? window : 1;
  a.local_start = window > 0 ? local_start : 0;
  a.n_local = n_local; a.n_chunks = n_chunks;
  a.part = static_cast<float*>(workspace);
  a.out = out; a.out_bf16 = out_dtype == LOUISKV_BF16; a.lse_out = lse_out;
  a.seg_state = seg_state; a.seg_stride = kSegRing + window; a.n_tokens = n_tokens;
  a.slice_div = slice_div;
  if (step_sync) {
    a.sync = *step_sync;
    a.step_waves = step_bf16 ? kStepAttnWaves : 0;
  }
  a.grid = (unsigned)(n_slices * n_chunks);
  // a chunk spans at most ceil(total / n_chunks) <= ceil((buf_rows + window) / n_chunks) rows
  a.lds = indexed ? (size_t)(((int64_t)buf_rows + window + n_chunks - 1) / n_chunks + 1) * sizeof(int) : 0;
  if (step_sync && n_chunks > 1)   // the merging block stages every chunk's (m, l) per head there
    a.lds = std::max(a.lds, (size_t)n_chunks * group_size * sizeof(float2));
  hipStream_t s = as_stream(stream);
  if (indexed)
    launch_attn<true>(dtype, group_size, a, s);
  else
    launch_attn<false>(dtype, group_size, a, s);
  LKV_CHECK_LAUNCH();
  if (n_chunks == 1 || step_sync) return LOUISKV_OK;     // the blocks wrote the output themselves
  const int64_t n_rows = n_slices * group_size;
  const int cgrid = (int)((n_rows + 3) / 4);
  if (out_dtype == LOUISKV_BF16)
    attn_combine_kernel<uint16_t><<<cgrid, 256, 0, s>>>(a.part, n_chunks, group_size, n_rows,
                                                        static_cast<uint16_t*>(out), lse_out);
  else
    attn_combine_kernel<float><<<cgrid, 256, 0, s>>>(a.part, n_chunks, group_size, n_rows, static_cast<float*>(out),
                                                     lse_out);
  LKV_CHECK_LAUNCH();
  return LOUISKV_OK;
}

}  // namespace
}  // namespace louiskv

extern "C" int louiskv_sparse_decode_attn(const void* q, int32_t dtype, int64_t n_slices, int32_t n_kv_heads,
                                          int32_t group_size, int32_t d, float scale, const void* k_buf,
                                          const void* v_buf, const int32_t* n_sel, int32_t buf_rows,
                                          const void* k_local, const void* v_local, int32_t window,
                                          int32_t local_start, int32_t n_local, void* out, int32_t out_dtype,
                                          float* lse_out, void* workspace, size_t workspace_bytes, void* stream) {
  return sparse_decode_attn(q, dtype, n_slices, n_kv_heads, group_size, d, scale, k_buf, v_buf, n_sel, buf_rows,
                            nullptr, buf_rows, k_local, v_local, window, local_start, n_local, out, out_dtype,
                            lse_out, workspace, workspace_bytes, stream);
}

extern "C" int louiskv_sparse_decode_attn_rows(const void* q, int32_t dtype, int64_t n_slices, int32_t n_kv_heads,
                                               int32_t group_size, int32_t d, float scale, const void* k_pool,
                                               const void* v_pool, int64_t pool_rows, const int32_t* sel_rows,
                                               const int32_t* n_sel, int32_t budget, const void* k_local,
                                               const void* v_local, int32_t window, int32_t local_start,
                                               int32_t n_local, void* out, int32_t out_dtype, float* lse_out,
                                               void* workspace, size_t workspace_bytes, void* stream) {
  if (!sel_rows) return fail(LOUISKV_ERR_NULL, "sel_rows is required");
  return sparse_decode_attn(q, dtype, n_slices, n_kv_heads, group_size, d, scale, k_pool, v_pool, n_sel, budget,
                            sel_rows, pool_rows, k_local, v_local, window, local_start, n_local, out, out_dtype,
                            lse_out, workspace, workspace_bytes, stream);
}

// ---------------------------------------------------------------------------
// One decode step of Algorithm 1 in one launch (bf16: step_fused_kernel) or
// two (float32, and with the LRU cache: step_select_kernel, then the
// attention) (fixed segments, KV_critical as a row list).

namespace louiskv {
namespace {

struct StepLayout {
  size_t counters, logits, pmax, fetch, part, total;
};

// Polls of the one-launch step's bounded wait: kStepSpinLimit, or fewer from
// LOUISKV_STEP_SPIN_LIMIT (tests of the time-out path).
int step_spin_limit() {
  const char* e = getenv("LOUISKV_STEP_SPIN_LIMIT");
  if (e && *e) {
    const long v = strtol(e, nullptr, 10);
    if (v >= 1 && v <= kStepSpinLimit) return (int)v;
  }
  return kStepSpinLimit;
}

// Workspace of a decode step: the arrival counters and flags (zero between
// calls; the one-launch step keeps selection and attention counters and
// ready flags per slice, group counters and a status word kStepSyncStride
// ints apart, the two-launch step its two counters per slice packed at the
// start), logits and part maxima, with a cached KV_critical the transfer
// plan's scratch (fetch slots, rows, counts), and the attention partials.
StepLayout step_layout(int64_t S, int dtype, int G, int units_cap, int budget, int window, bool cached = false) {
  StepLayout L{};
  Carver cv(nullptr);
  cv.take<int32_t>(((size_t)4 * S + 1) * kStepSyncStride);
  L.logits = align_up(cv.used, 256);
  cv.take<double>((size_t)S * units_cap * G);
  L.pmax = align_up(cv.used, 256);
  cv.take<double>((size_t)S * std::max(kMaxLogitParts, kMaxSelectParts) * G);
  L.fetch = align_up(cv.used, 256);
  if (cached) cv.take<int32_t>((size_t)S * (2 * (size_t)std::max(budget, 1) + 1));
  L.part = align_up(cv.used, 256);
  cv.take<char>(step_attn_part_bytes(S, G, budget, window, dtype));
  L.counters = 0;
  L.total = align_up(cv.used, 256);
  return L;
}

int plan_and_fetch(const int32_t* row_ws, const int32_t* n_sel, const uint8_t* fire, int64_t n_slices,
                   int32_t n_kv_heads, int32_t budget, int32_t cache_rows, int64_t pool_rows, int32_t step,
                   int32_t* buf_row, int32_t* slot_step, int32_t* slot_list, int32_t* fslot, int32_t* frow,
                   int32_t* nfetch, int32_t* n_fetched, int32_t dtype, const void* kpd, const void* vpd, void* k_buf,
                   void* v_buf, hipStream_t s);

// KV_critical kept as an LRU cache of pool rows (louiskv_decode_step_cached).
struct StepCache {
  int32_t pool_on_host, cache_rows;
  void *k_buf, *v_buf;
  int32_t *buf_row, *slot_step, *slot_list, *n_fetched;
};

}  // namespace
}  // namespace louiskv

extern "C" size_t louiskv_decode_step_workspace_size(int64_t n_slices, int32_t dtype, int32_t group_size,
                                                     int32_t units_cap, int32_t budget, int32_t window) {
  if (n_slices < 1 || group_size < 1 || group_size > kMaxGroupSize || units_cap < 1 || budget < 0 || window < 0 ||
      (dtype != LOUISKV_F32 && dtype != LOUISKV_BF16))
    return 0;
  return step_layout(n_slices, dtype, group_size, units_cap, budget, window).total;
}

namespace louiskv {
namespace {
int decode_step_impl(const void* q, void* q_ref, int32_t dtype, int64_t n_groups, int32_t n_q_heads,
                     int32_t n_kv_heads, int32_t d, double tau, int32_t mode, int32_t step, double* r_out,
                     uint8_t* fire_out, const void* k_new, const void* v_new, void* k_local, void* v_local,
                     int32_t window, int32_t seg_len, float* reps, int32_t* unit_start, int32_t* unit_size,
                     int32_t units_cap, int32_t n_clusters, void* k_pool, void* v_pool, int64_t pool_rows,
                     int32_t prompt_len, int32_t budget, int32_t* sel_units, int32_t* n_sel_units, int32_t* n_sel,
                     int32_t* sel_rows, double* scores_out, void* out, int32_t out_dtype, float* lse_out,
                     void* workspace, size_t workspace_bytes, void* stream, const StepCache* cache) {
  if (!q || !q_ref || !fire_out || !k_new || !v_new || !k_local || !v_local || !out)
    return fail(LOUISKV_ERR_NULL, "q, q_ref, fire_out, k_new, v_new, k_local, v_local and out are required");
  if (!reps || !unit_start || !unit_size || !k_pool || !v_pool || !sel_units || !n_sel_units || !n_sel || !sel_rows)
    return fail(LOUISKV_ERR_NULL, "unit tables, pools and selection outputs are required");
  int st = check_dtype(dtype);
  if (st) return st;
  if ((st = check_dtype(out_dtype))) return st;
  if (d != kHeadDim) return fail(LOUISKV_ERR_UNSUPPORTED, "head dim %d not supported (only 128)", d);
  if (n_kv_heads < 1 || n_groups < 1 || n_q_heads < 1 || n_q_heads % n_kv_heads != 0 ||
      n_groups * n_kv_heads > INT32_MAX)
    return fail(LOUISKV_ERR_SHAPE, "n_groups=%lld n_q_heads=%d n_kv_heads=%d", (long long)n_groups, n_q_heads,
                n_kv_heads);
  const int group_size = n_q_heads / n_kv_heads;
  if (group_size != 1 && group_size != 2 && group_size != 4 && group_size != 8)
    return fail(LOUISKV_ERR_UNSUPPORTED, "group_size=%d must be 1, 2, 4 or 8", group_size);
  if (mode != LOUISKV_REF_PREV && mode != LOUISKV_REF_ANCHOR) return fail(LOUISKV_ERR_SHAPE, "unknown mode %d", mode);
  if (budget < 0 || prompt_len < 0 || n_clusters < 1) 
    return fail(LOUISKV_ERR_SHAPE, "budget=%d prompt_len=%d n_clusters=%d", budget, prompt_len, n_clusters);
  int32_t ev = -1, n_ev = 0, n_local = 0, local_start = 0;
  if ((st = louiskv_window_info(step, window, seg_len, &ev, &n_ev, &n_local, &local_start))) return st;
  // units scorable at this step: the clusters and the segments evicted before it
  int32_t n_ev_before = 0;
  if (step > 0 && (st = louiskv_window_info(step - 1, window, seg_len, nullptr, &n_ev_before, nullptr, nullptr)))
    return st;
  const int64_t n_units = (int64_t)n_clusters + n_ev_before;
  if (n_units > units_cap || n_units > kMaxUnits || (ev >= 0 && (int64_t)n_clusters + ev >= units_cap))
    return fail(LOUISKV_ERR_SHAPE, "units %lld (and an evicted one) exceed units_cap=%d (at most %d)",
                (long long)n_units, units_cap, kMaxUnits);
  if ((int64_t)prompt_len + (int64_t)(ev + 1) * seg_len > pool_rows || pool_rows < 1)
    return fail(LOUISKV_ERR_SHAPE, "segment rows exceed pool_rows=%lld", (long long)pool_rows);
  const int64_t n_slices = n_groups * n_kv_heads;
  void* kpd = k_pool;
  void* vpd = v_pool;
  if (cache) {
    if (!cache->k_buf || !cache->v_buf || !cache->buf_row || !cache->slot_step || !cache->slot_list)
      return fail(LOUISKV_ERR_NULL, "k_buf, v_buf, buf_row, slot_step and slot_list are required");
    if (budget < 1 || cache->cache_rows < budget || cache->cache_rows > kCacheMaxRows)
      return fail(LOUISKV_ERR_SHAPE, "cache_rows=%d must be in [budget=%d, %d]", cache->cache_rows, budget,
                  kCacheMaxRows);
    if (step > kCacheMaxStep) return fail(LOUISKV_ERR_SHAPE, "step=%d must be at most %d", step, kCacheMaxStep);
    if (pool_rows > kDeltaMaxPoolRows)
      return fail(LOUISKV_ERR_UNSUPPORTED, "pool_rows=%lld must be at most %lld", (long long)pool_rows,
                  (long long)kDeltaMaxPoolRows);
    if (cache->pool_on_host &&
        ((st = device_view_of_host_pool(k_pool, &kpd)) || (st = device_view_of_host_pool(v_pool, &vpd))))
      return st;
  }
  const StepLayout lay = step_layout(n_slices, dtype, group_size, units_cap, budget, window, cache != nullptr);
  if (!workspace || workspace_bytes < lay.total)
    return fail(LOUISKV_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", lay.total, workspace_bytes);
  char* ws = static_cast<char*>(workspace);
  int32_t* sel_counter = reinterpret_cast<int32_t*>(ws + lay.counters);
  int32_t* attn_counter = sel_counter + n_slices;
  double* logit_ws = reinterpret_cast<double*>(ws + lay.logits);
  double* part_max = reinterpret_cast<double*>(ws + lay.pmax);
  const int n_parts = logit_parts(n_slices, (int)n_units);
  int n_pad = 64;
  while (n_pad < n_units) n_pad <<= 1;
  const size_t lds = (size_t)n_pad * (sizeof(uint64_t) + 2 * sizeof(int));
  const double scale = 1.0 / sqrt((double)kHeadDim);
  hipStream_t s = as_stream(stream);
  if (!cache && dtype == LOUISKV_BF16) {   // the whole step in one launch
    // blocks per slice: one per kStepAttnRows rows (a 16-row tile per wave),
    // at most kStepMaxBlocks, and at most one block per compute unit over the
    // launch (a block of the selection's register footprint fills one), so
    // that every block can be resident at once whenever blocks wait (two or
    // more per slice; a slice's only block never waits)
    const int cus = device_cu_count();
    const int64_t step_cus = cus > 0 ? cus : 256;
    const int nb = (int)std::max<int64_t>(
        1, std::min<int64_t>({(int64_t)kStepMaxBlocks, (int64_t)step_attn_chunks(budget, window),
                              step_cus / n_slices}));
    const int64_t total_rows = (int64_t)budget + window;
    const int chunk_rows = (int)(((total_rows + nb - 1) / nb + 15) / 16 * 16);
    if (n_slices * nb > INT32_MAX) return fail(LOUISKV_ERR_SHAPE, "problem too large for one launch");
    FusedStep fa{};
    fa.q = static_cast<const uint16_t*>(q);
    fa.q_ref = static_cast<uint16_t*>(q_ref);
    fa.n_slices = n_slices;
    fa.n_kv_heads = n_kv_heads;
    fa.first = step == 0 ? 1 : 0;
    fa.mode = mode;
    fa.tau = tau;
    fa.r_out = r_out;
    fa.fire_out = fire_out;
    fa.k_new = static_cast<const uint16_t*>(k_new);
    fa.v_new = static_cast<const uint16_t*>(v_new);
    fa.k_local = static_cast<uint16_t*>(k_local);
    fa.v_local = static_cast<uint16_t*>(v_local);
    fa.window = window;
    fa.step = step;
    fa.seg_len = seg_len;
    fa.evict_seg = ev;
    fa.reps = reps;
    fa.unit_start = unit_start;
    fa.unit_size = unit_size;
    fa.units_cap = units_cap;
    fa.n_clusters = n_clusters;
    fa.k_pool = static_cast<uint16_t*>(k_pool);
    fa.v_pool = static_cast<uint16_t*>(v_pool);
    fa.pool_rows = pool_rows;
    fa.prompt_len = prompt_len;
    fa.scale = scale;
    fa.n_units = (int)n_units;
    fa.budget = budget;
    fa.sel_units = sel_units;
    fa.n_sel_units = n_sel_units;
    fa.n_sel = n_sel;
    fa.sel_rows = sel_rows;
    fa.scores_out = scores_out;
    fa.logit_ws = logit_ws;
    fa.part_max = part_max;
    fa.sel_counter = sel_counter;
    fa.attn_counter = sel_counter + n_slices * kStepSyncStride;
    fa.ready = sel_counter + 2 * n_slices * kStepSyncStride;
    fa.grp_counter = sel_counter + 3 * n_slices * kStepSyncStride;
    fa.status = sel_counter + 4 * n_slices * kStepSyncStride;
    fa.n_blk = nb;
    fa.chunk_rows = chunk_rows;
    fa.n_pad = n_pad;
    fa.spin_limit = step_spin_limit();
    fa.local_start = local_start;
    fa.n_local = n_local;
    fa.part = reinterpret_cast<float*>(ws + lay.part);
    fa.out = out;
    fa.out_bf16 = out_dtype == LOUISKV_BF16;
    fa.lse_out = lse_out;
    const unsigned fgrid = (unsigned)(n_slices * nb);
#define LKV_STEP_FUSED(G)                                                                                   \
  {                                                                                                         \
    const size_t flds = std::max(lds, fused_attn_lds<G>(nb, chunk_rows));                                   \
    if ((st = check_lds(reinterpret_cast<const void*>(&step_fused_kernel<G>), flds))) return st;            \
    step_fused_kernel<G><<<fgrid, kSelThreads, flds, s>>>(fa);                                              \
  }
    switch (group_size) {
      case 1: LKV_STEP_FUSED(1); break;
      case 2: LKV_STEP_FUSED(2); break;
      case 4: LKV_STEP_FUSED(4); break;
      default: LKV_STEP_FUSED(8); break;
    }
#undef LKV_STEP_FUSED
    LKV_CHECK_LAUNCH();
    return LOUISKV_OK;
  }
  const unsigned grid = (unsigned)(n_slices * n_parts);
#define LKV_STEP_SEL(T, G)                                                                                           \
  if ((st = check_lds(reinterpret_cast<const void*>(&step_select_kernel<T, G>), lds))) return st;                    \
  step_select_kernel<T, G><<<grid, kSelThreads, lds, s>>>(                                                           \
      static_cast<const T*>(q), static_cast<const T*>(q_ref), n_kv_heads, tau, step == 0 ? 1 : 0, r_out, fire_out,  \
      static_cast<const T*>(k_new), static_cast<const T*>(v_new), static_cast<T*>(k_local), static_cast<T*>(v_local), \
      window, step, seg_len, ev, reps, unit_start, unit_size, units_cap, n_clusters, static_cast<T*>(kpd),           \
      static_cast<T*>(vpd), pool_rows, prompt_len, scale, (int)n_units, budget, sel_units, n_sel_units, n_sel,         \
      sel_rows, scores_out, logit_ws, part_max, sel_counter, n_parts, n_pad)
#define LKV_STEP_SEL_G(T)                   \
  switch (group_size) {                     \
    case 1: LKV_STEP_SEL(T, 1); break;      \
    case 2: LKV_STEP_SEL(T, 2); break;      \
    case 4: LKV_STEP_SEL(T, 4); break;      \
    default: LKV_STEP_SEL(T, 8); break;     \
  }
  if (dtype == LOUISKV_BF16) {
    LKV_STEP_SEL_G(uint16_t)
  } else {
    LKV_STEP_SEL_G(float)
  }
#undef LKV_STEP_SEL_G
#undef LKV_STEP_SEL
  LKV_CHECK_LAUNCH();
  const StepSync sync = {attn_counter, q_ref, fire_out, mode};
  if (!cache)
    return sparse_decode_attn(q, dtype, n_slices, n_kv_heads, group_size, d, (float)scale, k_pool, v_pool, n_sel,
                              budget, sel_rows, pool_rows, k_local, v_local, window, local_start, n_local, out,
                              out_dtype, lse_out, ws + lay.part, lay.total - lay.part, stream, nullptr, 0, 1, &sync);
  // the fired slices' selections (sel_rows) into the cache, then the
  // attention over the cached rows through the slot list
  int32_t* fslot = reinterpret_cast<int32_t*>(ws + lay.fetch);
  int32_t* frow = fslot + (size_t)n_slices * budget;
  int32_t* nfetch = frow + (size_t)n_slices * budget;
  if ((st = plan_and_fetch(sel_rows, n_sel, fire_out, n_slices, n_kv_heads, budget, cache->cache_rows, pool_rows,
                           step, cache->buf_row, cache->slot_step, cache->slot_list, fslot, frow, nfetch,
                           cache->n_fetched, dtype, kpd, vpd, cache->k_buf, cache->v_buf, s)))
    return st;
  return sparse_decode_attn(q, dtype, n_slices, n_kv_heads, group_size, d, (float)scale, cache->k_buf, cache->v_buf,
                            n_sel, budget, cache->slot_list, cache->cache_rows, k_local, v_local, window, local_start,
                            n_local, out, out_dtype, lse_out, ws + lay.part, lay.total - lay.part, stream, nullptr, 0, 1,
                            &sync);
}
}  // namespace
}  // namespace louiskv

extern "C" int louiskv_decode_step(const void* q, void* q_ref, int32_t dtype, int64_t n_groups, int32_t n_q_heads,
                                   int32_t n_kv_heads, int32_t d, double tau, int32_t mode, int32_t step,
                                   double* r_out, uint8_t* fire_out, const void* k_new, const void* v_new,
                                   void* k_local, void* v_local, int32_t window, int32_t seg_len, float* reps,
                                   int32_t* unit_start, int32_t* unit_size, int32_t units_cap, int32_t n_clusters,
                                   void* k_pool, void* v_pool, int64_t pool_rows, int32_t prompt_len, int32_t budget,
                                   int32_t* sel_units, int32_t* n_sel_units, int32_t* n_sel, int32_t* sel_rows,
                                   double* scores_out, void* out, int32_t out_dtype, float* lse_out,
                                   void* workspace, size_t workspace_bytes, void* stream) {
  return decode_step_impl(q, q_ref, dtype, n_groups, n_q_heads, n_kv_heads, d, tau, mode, step, r_out, fire_out, k_new,
                          v_new, k_local, v_local, window, seg_len, reps, unit_start, unit_size, units_cap, n_clusters,
                          k_pool, v_pool, pool_rows, prompt_len, budget, sel_units, n_sel_units, n_sel, sel_rows,
                          scores_out, out, out_dtype, lse_out, workspace, workspace_bytes, stream, nullptr);
}

extern "C" size_t louiskv_decode_step_cached_workspace_size(int64_t n_slices, int32_t dtype, int32_t group_size,
                                                            int32_t units_cap, int32_t budget, int32_t window) {
  if (n_slices < 1 || group_size < 1 || group_size > kMaxGroupSize || units_cap < 1 || budget < 1 || window < 0 ||
      (dtype != LOUISKV_F32 && dtype != LOUISKV_BF16))
    return 0;
  return step_layout(n_slices, dtype, group_size, units_cap, budget, window, true).total;
}

extern "C" int louiskv_decode_step_cached(
    const void* q, void* q_ref, int32_t dtype, int64_t n_groups, int32_t n_q_heads, int32_t n_kv_heads, int32_t d,
    double tau, int32_t mode, int32_t step, double* r_out, uint8_t* fire_out, const void* k_new, const void* v_new,
    void* k_local, void* v_local, int32_t window, int32_t seg_len, float* reps, int32_t* unit_start,
    int32_t* unit_size, int32_t units_cap, int32_t n_clusters, void* k_pool, void* v_pool, int64_t pool_rows,
    int32_t pool_on_host, int32_t prompt_len, int32_t budget, int32_t cache_rows, void* k_buf, void* v_buf,
    int32_t* buf_row, int32_t* slot_step, int32_t* slot_list, int32_t* n_fetched, int32_t* sel_units,
    int32_t* n_sel_units, int32_t* n_sel, int32_t* sel_rows, double* scores_out, void* out, int32_t out_dtype,
    float* lse_out, void* workspace, size_t workspace_bytes, void* stream) {
  const StepCache cache{pool_on_host, cache_rows, k_buf, v_buf, buf_row, slot_step, slot_list, n_fetched};
  return decode_step_impl(q, q_ref, dtype, n_groups, n_q_heads, n_kv_heads, d, tau, mode, step, r_out, fire_out, k_new,
                          v_new, k_local, v_local, window, seg_len, reps, unit_start, unit_size, units_cap, n_clusters,
                          k_pool, v_pool, pool_rows, prompt_len, budget, sel_units, n_sel_units, n_sel, sel_rows,
                          scores_out, out, out_dtype, lse_out, workspace, workspace_bytes, stream, &cache);
}


// ---------------------------------------------------------------------------
// Allocation-free attention over listed pool rows.  The split-KV partials live
// in a static device array instead of a caller workspace.  The array's name
// is only a host-side stand-in: host code uses the device address that
// hipGetSymbolAddress returns, looked up once per device.

static __device__ __align__(256) float scratch[LOUISKV_NOALLOC_SCRATCH_BYTES / sizeof(float)];

namespace louiskv {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};

// The current device's copy of `scratch`.
int scratch_on_current_device(void** addr) {
  int dev = -1;
  LKV_CHECK_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(LOUISKV_ERR_UNSUPPORTED, "device %d: the allocation-free calls serve devices 0..%d", dev,
                kMaxDevices - 1);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    LKV_CHECK_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(LOUISKV_ERR_HIP, "hipGetSymbolAddress gave no address for the scratch array");
    g_scratch_addr[dev] = p;
  }
  *addr = g_scratch_addr[dev];
  return LOUISKV_OK;
}

}  // namespace
}  // namespace louiskv

extern "C" int louiskv_sparse_decode_attn_rows_noalloc(const void* q, int32_t dtype, int64_t n_slices,
                                                       int32_t n_kv_heads, int32_t group_size, int32_t d,
                                                       float scale, const void* k_pool, const void* v_pool,
                                                       int64_t pool_rows, const int32_t* sel_rows,
                                                       const int32_t* n_sel, int32_t budget, const void* k_local,
                                                       const void* v_local, int32_t window, int32_t local_start,
                                                       int32_t n_local, void* out, int32_t out_dtype,
                                                       float* lse_out, void* stream) {
  if (!sel_rows) return fail(LOUISKV_ERR_NULL, "sel_rows is required");
  if (n_slices >= 1 && group_size >= 1 && budget >= 0 && window >= 0) {
    const size_t need = attn_ws_bytes(n_slices, group_size, budget, window, true);
    if (need > LOUISKV_NOALLOC_SCRATCH_BYTES)
      return fail(LOUISKV_ERR_WORKSPACE,
                  "the allocation-free call holds at most %zu bytes of partials and this launch needs %zu; "
                  "use louiskv_sparse_decode_attn_rows with a workspace",
                  (size_t)LOUISKV_NOALLOC_SCRATCH_BYTES, need);
  }
  void* ws = nullptr;
  const int st = scratch_on_current_device(&ws);
  if (st) return st;
  return sparse_decode_attn(q, dtype, n_slices, n_kv_heads, group_size, d, scale, k_pool, v_pool, n_sel, budget,
                            sel_rows, pool_rows, k_local, v_local, window, local_start, n_local, out, out_dtype,
                            lse_out, ws, LOUISKV_NOALLOC_SCRATCH_BYTES, stream);
}

extern "C" int louiskv_retrieve_rows_per_head(const void* q, int32_t dtype, int64_t n_slices, int32_t n_kv_heads,
                                              int32_t group_size, int32_t d, double scale, const float* reps,
                                              const int32_t* unit_start, const int32_t* unit_size, int32_t units_cap,
                                              int32_t n_units, int32_t budget, const uint8_t* fire,
                                              int32_t* sel_units, int32_t* n_sel_units, int32_t* n_sel,
                                              int32_t* sel_rows, double* scores_out, void* workspace,
                                              size_t workspace_bytes, void* stream) {
  int st = check_retrieve_common(q, dtype, n_slices, n_kv_heads, group_size, d, reps, unit_start, unit_size, units_cap,
                                 n_units, budget, sel_units, n_sel_units, n_sel);
  if (st) return st;
  if (budget > 0 && !sel_rows) return fail(LOUISKV_ERR_NULL, "sel_rows is required when budget > 0");
  // one list per query head: the scorer runs with groups of one over
  // n_slices * group_size lists, each reading its KV head's units
  const int64_t lists = n_slices * group_size;
  if (lists > INT32_MAX) return fail(LOUISKV_ERR_SHAPE, "problem too large for one launch");
  const size_t need = align_up(logit_ws_doubles(lists, units_cap) * sizeof(double), 256);
  if (!workspace || workspace_bytes < need)
    return fail(LOUISKV_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, workspace_bytes);
  return score_and_select(q, dtype, lists, n_kv_heads * group_size, 1, d, scale, reps, unit_start, unit_size,
                          units_cap, n_units, budget, fire, sel_units, n_sel_units, n_sel, sel_rows, scores_out,
                          static_cast<double*>(workspace), nullptr, 0, as_stream(stream), group_size);
}

extern "C" int louiskv_sparse_decode_attn_rows_per_head(const void* q, int32_t dtype, int64_t n_slices,
                                                        int32_t n_kv_heads, int32_t group_size, int32_t d,
                                                        float scale, const void* k_pool, const void* v_pool,
                                                        int64_t pool_rows, const int32_t* sel_rows,
                                                        const int32_t* n_sel, int32_t budget, const void* k_local,
                                                        const void* v_local, int32_t window, int32_t local_start,
                                                        int32_t n_local, void* out, int32_t out_dtype,
                                                        float* lse_out, void* workspace, size_t workspace_bytes,
                                                        void* stream) {
  if (!sel_rows) return fail(LOUISKV_ERR_NULL, "sel_rows is required");
  if (group_size < 1 || group_size > kMaxGroupSize)
    return fail(LOUISKV_ERR_UNSUPPORTED, "group_size=%d must be in [1, %d]", group_size, kMaxGroupSize);
  if (n_kv_heads < 1 || n_slices < 1 || n_slices % n_kv_heads != 0 || n_slices * group_size > INT32_MAX)
    return fail(LOUISKV_ERR_SHAPE, "n_slices=%lld must be a positive multiple of n_kv_heads=%d", (long long)n_slices,
                n_kv_heads);
  // one list per query head over its KV head's pool and window
  return sparse_decode_attn(q, dtype, n_slices * group_size, n_kv_heads * group_size, 1, d, scale, k_pool, v_pool,
                            n_sel, budget, sel_rows, pool_rows, k_local, v_local, window, local_start, n_local, out,
                            out_dtype, lse_out, workspace, workspace_bytes, stream, nullptr, 0, group_size);
}

extern "C" int louiskv_sparse_decode_attn_seg(const void* q, int32_t dtype, int64_t n_slices, int32_t n_kv_heads,
                                              int32_t group_size, int32_t d, float scale, const void* k_buf,
                                              const void* v_buf, const int32_t* n_sel, int32_t buf_rows,
                                              const void* k_local, const void* v_local, int32_t window,
                                              const int32_t* seg_state, int32_t n_tokens, void* out,
                                              int32_t out_dtype, float* lse_out, void* workspace,
                                              size_t workspace_bytes, void* stream) {
  int st = check_seg_state(seg_state, window);
  if (st) return st;
  if (n_tokens < 1) return fail(LOUISKV_ERR_SHAPE, "n_tokens=%d must be >= 1", n_tokens);
  return sparse_decode_attn(q, dtype, n_slices, n_kv_heads, group_size, d, scale, k_buf, v_buf, n_sel, buf_rows,
                            nullptr, buf_rows, k_local, v_local, window, 0, window, out, out_dtype, lse_out,
                            workspace, workspace_bytes, stream, seg_state, n_tokens);
}

extern "C" int louiskv_sparse_decode_attn_rows_seg(const void* q, int32_t dtype, int64_t n_slices,
                                                   int32_t n_kv_heads, int32_t group_size, int32_t d, float scale,
                                                   const void* k_pool, const void* v_pool, int64_t pool_rows,
                                                   const int32_t* sel_rows, const int32_t* n_sel, int32_t budget,
                                                   const void* k_local, const void* v_local, int32_t window,
                                                   const int32_t* seg_state, int32_t n_tokens, void* out,
                                                   int32_t out_dtype, float* lse_out, void* workspace,
                                                   size_t workspace_bytes, void* stream) {
  if (!sel_rows) return fail(LOUISKV_ERR_NULL, "sel_rows is required");
  int st = check_seg_state(seg_state, window);
  if (st) return st;
  if (n_tokens < 1) return fail(LOUISKV_ERR_SHAPE, "n_tokens=%d must be >= 1", n_tokens);
  return sparse_decode_attn(q, dtype, n_slices, n_kv_heads, group_size, d, scale, k_pool, v_pool, n_sel, budget,
                            sel_rows, pool_rows, k_local, v_local, window, 0, window, out, out_dtype, lse_out,
                            workspace, workspace_bytes, stream, seg_state, n_tokens);
}

extern "C" size_t louiskv_retrieve_delta_workspace_size(int64_t n_slices, int32_t units_cap, int32_t budget) {
  if (n_slices < 1 || units_cap < 1 || budget < 1) return 0;
  Carver cv(nullptr);
  cv.take<double>(logit_ws_doubles(n_slices, units_cap));
  cv.take<int32_t>((size_t)n_slices * budget);   // selected pool rows
  cv.take<int32_t>((size_t)n_slices * budget);   // fetch slots
  cv.take<int32_t>((size_t)n_slices * budget);   // fetch rows
  cv.take<int32_t>((size_t)n_slices);            // fetch counts
  return align_up(cv.used, 256);
}

namespace louiskv {
namespace {
// The transfer plan of the fired slices' selections (row_ws: [S][budget]
// pool rows, n_sel each) into the KV_critical buffers (slot_step: the LRU
// cache of cache_rows slots; null: the buffer holds the last selection) and
// the copy of the planned rows; fslot, frow [S][budget] and nfetch [S] are
// scratch.
int plan_and_fetch(const int32_t* row_ws, const int32_t* n_sel, const uint8_t* fire, int64_t n_slices,
                   int32_t n_kv_heads, int32_t budget, int32_t cache_rows, int64_t pool_rows, int32_t step,
                   int32_t* buf_row, int32_t* slot_step, int32_t* slot_list, int32_t* fslot, int32_t* frow,
                   int32_t* nfetch, int32_t* n_fetched, int32_t dtype, const void* kpd, const void* vpd, void* k_buf,
                   void* v_buf, hipStream_t s) {
  int st;
  const size_t lds = (size_t)((pool_rows + 31) / 32) * sizeof(uint32_t);
  if (slot_step) {
    // the smallest per-thread slot run that covers cache_rows
    const int per = (cache_rows + kPlanThreads - 1) / kPlanThreads;
    auto plan = per <= 8 ? &cache_plan_kernel<8> : per <= 16 ? &cache_plan_kernel<16>
              : per <= 32 ? &cache_plan_kernel<32> : &cache_plan_kernel<64>;
    if ((st = check_lds(reinterpret_cast<const void*>(plan), lds))) return st;
    plan<<<(unsigned)n_slices, kPlanThreads, lds, s>>>(row_ws, n_sel, fire, n_kv_heads, budget, cache_rows, pool_rows,
                                                       step, buf_row, slot_step, slot_list, fslot, frow, nfetch,
                                                       n_fetched);
  } else {
    if ((st = check_lds(reinterpret_cast<const void*>(&delta_plan_kernel), lds))) return st;
    delta_plan_kernel<<<(unsigned)n_slices, kPlanThreads, lds, s>>>(row_ws, n_sel, fire, n_kv_heads, budget,
                                                                    pool_rows, buf_row, slot_list, fslot, frow, nfetch,
                                                                    n_fetched);
  }
  LKV_CHECK_LAUNCH();
  const int rpb = 128;
  const int bps = (budget + rpb - 1) / rpb;
  const unsigned grid = (unsigned)(n_slices * bps);
  if (dtype == LOUISKV_BF16)
    delta_fetch_kernel<uint16_t><<<grid, 256, 0, s>>>(static_cast<const uint16_t*>(kpd),
                                                      static_cast<const uint16_t*>(vpd), pool_rows, fslot, frow, nfetch,
                                                      budget, bps, rpb, static_cast<uint16_t*>(k_buf),
                                                      static_cast<uint16_t*>(v_buf), cache_rows);
  else
    delta_fetch_kernel<float><<<grid, 256, 0, s>>>(static_cast<const float*>(kpd), static_cast<const float*>(vpd),
                                                   pool_rows, fslot, frow, nfetch, budget, bps, rpb,
                                                   static_cast<float*>(k_buf), static_cast<float*>(v_buf), cache_rows);
  LKV_CHECK_LAUNCH();
  return LOUISKV_OK;
}

// Scores and selection, then the transfer plan (delta: the buffer holds the
// last selection only; cached: an LRU cache of cache_rows pool rows) and the
// fetch of the planned rows.
int retrieve_into_buffer(const void* q, int32_t dtype, int64_t n_slices, int32_t n_kv_heads, int32_t group_size,
                         int32_t d, double scale, const float* reps, const int32_t* unit_start,
                         const int32_t* unit_size, int32_t units_cap, int32_t n_units, const int32_t* seg_state,
                         int32_t window, const void* k_pool, const void* v_pool, int64_t pool_rows,
                         int32_t pool_on_host, int32_t budget, int32_t cache_rows, int32_t step,
                         const uint8_t* fire, int32_t* sel_units, int32_t* n_sel_units, int32_t* n_sel, void* k_buf,
                         void* v_buf, int32_t* buf_row, int32_t* slot_step, int32_t* slot_list, int32_t* n_fetched,
                         double* scores_out, void* workspace, size_t workspace_bytes, void* stream) {
  int st = check_retrieve_common(q, dtype, n_slices, n_kv_heads, group_size, d, reps, unit_start, unit_size, units_cap,
                                 n_units, budget, sel_units, n_sel_units, n_sel);
  if (st) return st;
  if (!k_pool || !v_pool || !k_buf || !v_buf || !buf_row || !slot_list)
    return fail(LOUISKV_ERR_NULL, "k_pool, v_pool, k_buf, v_buf, buf_row and slot_list are required");
  if (budget < 1) return fail(LOUISKV_ERR_SHAPE, "budget=%d must be >= 1", budget);
  if (cache_rows < budget) return fail(LOUISKV_ERR_SHAPE, "cache_rows=%d < budget=%d", cache_rows, budget);
  if (slot_step && cache_rows > kCacheMaxRows)
    return fail(LOUISKV_ERR_UNSUPPORTED, "cache_rows=%d exceeds %d", cache_rows, kCacheMaxRows);
  if (slot_step && (step < 0 || step > kCacheMaxStep))
    return fail(LOUISKV_ERR_SHAPE, "step=%d must be in [0, %d]", step, kCacheMaxStep);
  if (pool_rows < 1 || pool_rows > kDeltaMaxPoolRows)
    return fail(LOUISKV_ERR_UNSUPPORTED, "pool_rows=%lld must be in [1, %lld]", (long long)pool_rows,
                (long long)kDeltaMaxPoolRows);
  if (seg_state && (st = check_seg_state(seg_state, window))) return st;
  void* kpd = const_cast<void*>(k_pool);
  void* vpd = const_cast<void*>(v_pool);
  if (pool_on_host && ((st = device_view_of_host_pool(k_pool, &kpd)) || (st = device_view_of_host_pool(v_pool, &vpd))))
    return st;
  const size_t need = louiskv_retrieve_delta_workspace_size(n_slices, units_cap, budget);
  if (!workspace || workspace_bytes < need)
    return fail(LOUISKV_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, workspace_bytes);
  Carver cv(workspace);
  double* logit_ws = cv.take<double>(logit_ws_doubles(n_slices, units_cap));
  int32_t* row_ws = cv.take<int32_t>((size_t)n_slices * budget);
  int32_t* fslot = cv.take<int32_t>((size_t)n_slices * budget);
  int32_t* frow = cv.take<int32_t>((size_t)n_slices * budget);
  int32_t* nfetch = cv.take<int32_t>((size_t)n_slices);
  hipStream_t s = as_stream(stream);
  if ((st = score_and_select(q, dtype, n_slices, n_kv_heads, group_size, d, scale, reps, unit_start, unit_size,
                             units_cap, n_units, budget, fire, sel_units, n_sel_units, n_sel, row_ws, scores_out,
                             logit_ws, seg_state, seg_state ? kSegRing + window : 0, s)))
    return st;
  return plan_and_fetch(row_ws, n_sel, fire, n_slices, n_kv_heads, budget, cache_rows, pool_rows, step, buf_row,
                        slot_step, slot_list, fslot, frow, nfetch, n_fetched, dtype, kpd, vpd, k_buf, v_buf, s);
}
}  // namespace
}  // namespace louiskv

extern "C" int louiskv_retrieve_delta(const void* q, int32_t dtype, int64_t n_slices, int32_t n_kv_heads,
                                      int32_t group_size, int32_t d, double scale, const float* reps,
                                      const int32_t* unit_start, const int32_t* unit_size, int32_t units_cap,
                                      int32_t n_units, const int32_t* seg_state, int32_t window,
                                      const void* k_pool, const void* v_pool, int64_t pool_rows,
                                      int32_t pool_on_host, int32_t budget, const uint8_t* fire,
                                      int32_t* sel_units, int32_t* n_sel_units, int32_t* n_sel, void* k_buf,
                                      void* v_buf, int32_t* buf_row, int32_t* slot_list, int32_t* n_fetched,
                                      double* scores_out, void* workspace, size_t workspace_bytes, void* stream) {
  return retrieve_into_buffer(q, dtype, n_slices, n_kv_heads, group_size, d, scale, reps, unit_start, unit_size,
                              units_cap, n_units, seg_state, window, k_pool, v_pool, pool_rows, pool_on_host, budget,
                              budget, 0, fire, sel_units, n_sel_units, n_sel, k_buf, v_buf, buf_row, nullptr,
                              slot_list, n_fetched, scores_out, workspace, workspace_bytes, stream);
}

extern "C" int louiskv_retrieve_cached(const void* q, int32_t dtype, int64_t n_slices, int32_t n_kv_heads,
                                       int32_t group_size, int32_t d, double scale, const float* reps,
                                       const int32_t* unit_start, const int32_t* unit_size, int32_t units_cap,
                                       int32_t n_units, const int32_t* seg_state, int32_t window,
                                       const void* k_pool, const void* v_pool, int64_t pool_rows,
                                       int32_t pool_on_host, int32_t budget, int32_t cache_rows, int32_t step,
                                       const uint8_t* fire, int32_t* sel_units, int32_t* n_sel_units,
                                       int32_t* n_sel, void* k_buf, void* v_buf, int32_t* buf_row,
                                       int32_t* slot_step, int32_t* slot_list, int32_t* n_fetched,
                                       double* scores_out, void* workspace, size_t workspace_bytes, void* stream) {
  if (!slot_step) return fail(LOUISKV_ERR_NULL, "slot_step is required");
  return retrieve_into_buffer(q, dtype, n_slices, n_kv_heads, group_size, d, scale, reps, unit_start, unit_size,
                              units_cap, n_units, seg_state, window, k_pool, v_pool, pool_rows, pool_on_host, budget,
                              cache_rows, step, fire, sel_units, n_sel_units, n_sel, k_buf, v_buf, buf_row, slot_step,
                              slot_list, n_fetched, scores_out, workspace, workspace_bytes, stream);
}
