// Prefill-stage k-means of prompt keys (Section 4.2 prefill stage; Algorithm 1
// store_cache prefill branch), one independent problem per (sequence, layer,
// KV head) slice.
//
// Per Lloyd iteration:
//   prep     centroid operand for the matrix cores: -2 * op(c) laid out as MFMA
//            A-fragments (op = bf16 RNE rounding for bf16 keys, identity for fp32),
//            plus ||op(c)||^2 (float64 sum, rounded to fp32); zero the counts.
//   assign   D = ||op(c)||^2 - 2 op(c).k on MFMA (the norm enters as the
//            accumulator input), running argmin per key kept in registers,
//            block histogram of the chosen clusters into counts.
//   scan     exclusive scan of counts -> CSR offsets and scatter cursors.
//   scatter  key ids into their cluster's member range (order unspecified).
//   sum      centroid = float64 sum of members / count, rounded once to fp32;
//            empty clusters keep their centroid.  Sums of bf16 or fp32 inputs
//            are exact in float64 at these sizes, so the order is irrelevant.
//            The same kernel writes the next iteration's operand and clears
//            the counts (prep runs once, before the first iteration).
// From the second iteration on, the assignment starts each key's running
// minimum at a bound from its previous centroid, so the index search runs
// only for tiles that hold a closer centroid.
// After the last iteration, finalize sorts each member range ascending (the
// perm output), writes the unit table, and pack copies K/V rows into the pool.
#include "common.h"

namespace louiskv {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float floatx16;

constexpr int kTileC = 32;                 // centroids per MFMA tile (rows of D)
constexpr int kBf16Steps = 8;              // 32x32x16 MFMAs per 128-wide dot product
constexpr int kBf16TileU4 = kBf16Steps * 64;       // uint4 per bf16 operand tile (8 KB)
constexpr int kF32TileU4 = 16 * 64;                // uint4 per fp32 operand tile (16 KB)

#ifndef LKV_BF16_KEY_TILES
#define LKV_BF16_KEY_TILES 4
#endif
#ifndef LKV_BF16_STAGE_TILES
#define LKV_BF16_STAGE_TILES 2
#endif
#ifndef LKV_ASSIGN_WAVES
#define LKV_ASSIGN_WAVES 4
#endif
constexpr int kAssignThreads = 256;                          // fp32 kernel block
constexpr int kBf16Waves = LKV_ASSIGN_WAVES;                 // waves sharing one LDS stage
constexpr int kBf16Threads = 64 * kBf16Waves;
constexpr int kBf16KeyTiles = LKV_BF16_KEY_TILES;            // 32-key tiles held per wave
constexpr int kBf16KeysPerBlock = kBf16Waves * 32 * kBf16KeyTiles;
constexpr int kBf16StageTiles = LKV_BF16_STAGE_TILES;        // centroid tiles per LDS stage
constexpr int kF32KeysPerBlock = 4 * 32;           // one 32-key tile per wave
constexpr int kF32StageTiles = 2;

__host__ __device__ inline int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Workgroups are dealt to the 8 XCDs round-robin by block id.  Renumber the
// first 8*floor(n/8) blocks so that consecutive logical blocks (the blocks of
// one slice) run on the same XCD and share its L2; the tail keeps its id.
constexpr int kXcds = 8;
__device__ __forceinline__ int xcd_local_block(int b, int n) {
  const int q = n / kXcds;
  if (b >= q * kXcds) return b;
  return (b % kXcds) * q + b / kXcds;
}

template <class T>
__global__ void init_centroids_kernel(const T* __restrict__ keys, const int32_t* __restrict__ init_idx,
                                      float* __restrict__ reps, int n_tokens, int n_clusters,
                                      int units_cap, int64_t n_rows) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n_rows) return;
  const int lane = threadIdx.x & 63;
  const int64_t s = row / n_clusters;
  const int c = (int)(row - s * n_clusters);
  int t = init_idx[s * n_clusters + c];
  t = t < 0 ? 0 : (t >= n_tokens ? n_tokens - 1 : t);
  const T* src = keys + ((size_t)s * n_tokens + t) * kHeadDim;
  float* dst = reps + ((size_t)s * units_cap + c) * kHeadDim;
  dst[2 * lane] = load_as_f32(src, 2 * lane);
  dst[2 * lane + 1] = load_as_f32(src, 2 * lane + 1);
}

// One wave per padded centroid row.  Writes the A-fragments of -2*op(c) and
// ||op(c)||^2; padding rows get a zero operand and +inf norm so they never win.
//
// Dimension k of a centroid maps to MFMA operand position (lane half h, step,
// element): bf16: k = 64h + 8*step + e; fp32: k = 64h + step.  The key operand
// uses the same map, so each product pairs equal dimensions.
template <bool kBf16>
__global__ void prep_operand_kernel(const float* __restrict__ reps, int units_cap, int n_clusters,
                                    int n_ctiles, uint4* __restrict__ frag, float* __restrict__ cnorm,
                                    int32_t* __restrict__ counts, int64_t n_rows) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n_rows) return;
  const int lane = threadIdx.x & 63;
  const int cpad = n_ctiles * kTileC;
  const int64_t s = row / cpad;
  const int c = (int)(row - s * cpad);
  const bool real = c < n_clusters;
  float v0 = 0.f, v1 = 0.f;
  if (real) {
    const float* src = reps + ((size_t)s * units_cap + c) * kHeadDim;
    v0 = src[2 * lane];
    v1 = src[2 * lane + 1];
  }
  if (kBf16) {
    v0 = bf16_to_f32(f32_to_bf16(v0));
    v1 = bf16_to_f32(f32_to_bf16(v1));
  }
  double nrm = wave_sum((double)v0 * v0 + (double)v1 * v1);
  const int t = c / kTileC, ci = c % kTileC;
  const int k0 = 2 * lane, h = k0 >> 6;
  const int flane = h * 32 + ci;
  if (kBf16) {
    const int step = (k0 & 63) >> 3, e = k0 & 7;
    uint16_t* f = reinterpret_cast<uint16_t*>(frag + ((size_t)s * n_ctiles + t) * kBf16TileU4);
    const uint32_t lo = f32_to_bf16(-2.f * v0), hi = f32_to_bf16(-2.f * v1);
    *reinterpret_cast<uint32_t*>(f + ((size_t)(step * 64 + flane) * 8 + e)) = lo | (hi << 16);
  } else {
    float* f = reinterpret_cast<float*>(frag + ((size_t)s * n_ctiles + t) * kF32TileU4);
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int step = (k0 + q) & 63;
      f[((size_t)(step >> 2) * 64 + flane) * 4 + (step & 3)] = -2.f * (q ? v1 : v0);
    }
  }
  if (lane == 0) {
    cnorm[(size_t)s * cpad + c] = real ? (float)nrm : __builtin_inff();
    if (real && counts) counts[(size_t)s * n_clusters + c] = 0;
  }
}

// Block histogram of chosen clusters, merged into counts[slice][*].
__device__ __forceinline__ void block_histogram(int* hist, bool lds_ok, int n_clusters, int32_t* counts_slice,
                                                const int* idx, const bool* valid, int n_local) {
  const int tid = threadIdx.x;
  if (lds_ok) {
    for (int i = tid; i < n_clusters; i += blockDim.x) hist[i] = 0;
    __syncthreads();
    for (int q = 0; q < n_local; ++q)
      if (valid[q]) atomicAdd(&hist[idx[q]], 1);
    __syncthreads();
    for (int i = tid; i < n_clusters; i += blockDim.x)
      if (hist[i]) atomicAdd(&counts_slice[i], hist[i]);
  } else {
    for (int q = 0; q < n_local; ++q)
      if (valid[q]) atomicAdd(&counts_slice[idx[q]], 1);
  }
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;

constexpr int kBf16Ring = 4;                          // LDS stage buffers in flight
constexpr int kBf16StageBytes = kBf16StageTiles * kBf16TileU4 * 16 + 64 * 4;
// DMA instructions each wave issues per stage: its share of the operand tiles
// plus one copy of the stage's norms (every wave writes the same norms, so the
// count is the same for all waves and vmcnt thresholds are uniform).
constexpr int kBf16DmaPerWave = kBf16StageTiles * (kBf16TileU4 / 64) / kBf16Waves + 1;
static_assert(kBf16StageTiles * (kBf16TileU4 / 64) % kBf16Waves == 0, "operand copies must split evenly");
static_assert(kBf16StageTiles * kTileC <= 64, "one 64-lane copy carries a stage's norms");

// Asynchronous copy of stage `st` (centroid operand tiles and their norms)
// straight from global memory into an LDS stage buffer; 64 lanes x 16 bytes
// per instruction, completion tracked by vmcnt.  The tile count is padded to
// whole stages, so every stage copies the same amount.
// Copies [q0, q1) of the wave's kBf16DmaPerWave instructions for stage st
// (the last one carries the norms), so a stage's copy can be spread out.
//
// The copies are written as inline assembly (scalar base address, per-lane
// offset, LDS destination in M0) rather than with the compiler builtin: the
// builtin makes the compiler track the LDS writes itself, and at the loop
// header it cannot tell the ring buffers apart and drains every copy in
// flight (vmcnt(0)) once per pass of the ring.  Written this way the compiler
// sees no memory operation, and the sweep's explicit vmcnt waits and barriers
// are the only synchronisation, as intended.
__device__ __forceinline__ void dma_16b(const void* base, uint32_t lane_off, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(lane_off), "s"(base), "s"(lds_addr)
               : "memory", "m0");
}
__device__ __forceinline__ void dma_4b(const void* base, uint32_t lane_off, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dword %0, %1" ::"v"(lane_off), "s"(base), "s"(lds_addr)
               : "memory", "m0");
}

__device__ __forceinline__ void stage_async_part(const uint4* fslice, const float* cslice, int st, char* buf,
                                                 int wave, int lane, int q0, int q1) {
  const uint4* src = fslice + (size_t)st * kBf16StageTiles * kBf16TileU4;
#pragma unroll
  for (int q = 0; q < kBf16DmaPerWave - 1; ++q) {
    if (q < q0 || q >= q1) continue;
    const int i = wave + q * kBf16Waves;   // wave-uniform
    dma_16b(src + i * 64, lane * 16, (uint32_t)(uintptr_t)(buf + i * 1024));
  }
  if (q1 == kBf16DmaPerWave) {
    const int c = lane % (kBf16StageTiles * kTileC);
    dma_4b(cslice + st * kBf16StageTiles * kTileC, c * 4,
           (uint32_t)(uintptr_t)(buf + kBf16StageTiles * kBf16TileU4 * 16));
  }
}

__device__ __forceinline__ void stage_async(const uint4* fslice, const float* cslice, int st, char* buf, int wave,
                                            int lane) {
  stage_async_part(fslice, cslice, st, buf, wave, lane, 0, kBf16DmaPerWave);
}

__device__ __forceinline__ void wait_vm_stages(int k) {
  // at most k later stages' copies may still be in flight
  if (k >= 2) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * kBf16DmaPerWave) : "memory");
  else if (k == 1) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kBf16DmaPerWave) : "memory");
  else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// Tile epilogue of the running argmin.  The lane's 16 results of a tile
// (rows ascending with v) are reduced to their minimum with min3 (8 ops); only
// when that beats the running best does the lane search for the lowest row
// holding it.  Because tiles are visited in ascending order and only a
// strictly smaller value replaces the best, the result is the lowest index
// among equal minima.  The search is skipped by a wave-uniform branch (taken
// when any lane improved) and applied with per-lane selects, so EXEC is never
// narrowed while matrix instructions are in flight.
// Row of result register v within the lane's half of a 32x32 tile.
#define LKV_ROW(v) (8 * ((v) >> 2) + ((v) & 3))

__device__ __forceinline__ float tile_min(const floatx16& x) {
  const float a = __builtin_fminf(__builtin_fminf(x[0], x[1]), x[2]);
  const float b = __builtin_fminf(__builtin_fminf(x[3], x[4]), x[5]);
  const float c = __builtin_fminf(__builtin_fminf(x[6], x[7]), x[8]);
  const float d = __builtin_fminf(__builtin_fminf(x[9], x[10]), x[11]);
  const float e = __builtin_fminf(__builtin_fminf(x[12], x[13]), x[14]);
  const float f = __builtin_fminf(__builtin_fminf(a, b), c);
  const float g = __builtin_fminf(__builtin_fminf(d, e), x[15]);
  return __builtin_fminf(f, g);
}

// Lowest row of the tile holding the value m (the lane's minimum).  All
// compares go first, each into its own SGPR pair, then the selects from the
// highest row down; written as a plain select chain the compiler pairs every
// compare with its select through VCC and pads each pair with wait states.
#define LKV_CMP(v) asm("v_cmp_eq_f32_e64 %0, %1, %2" : "=s"(e##v) : "v"(x[v]), "v"(m))
#define LKV_CND(v, row) asm("v_cndmask_b32_e64 %0, %1, " #row ", %2" : "=v"(id) : "v"(id), "s"(e##v))
__device__ __forceinline__ int tile_find(const floatx16& x, float m) {
  uint64_t e0, e1, e2, e3, e4, e5, e6, e7, e8, e9, e10, e11, e12, e13, e14;
  LKV_CMP(0); LKV_CMP(1); LKV_CMP(2); LKV_CMP(3); LKV_CMP(4); LKV_CMP(5); LKV_CMP(6); LKV_CMP(7);
  LKV_CMP(8); LKV_CMP(9); LKV_CMP(10); LKV_CMP(11); LKV_CMP(12); LKV_CMP(13); LKV_CMP(14);
  int id = LKV_ROW(15);
  // rows LKV_ROW(14..0) = 26 25 24 19 18 17 16 11 10 9 8 3 2 1 0
  LKV_CND(14, 26); LKV_CND(13, 25); LKV_CND(12, 24); LKV_CND(11, 19); LKV_CND(10, 18); LKV_CND(9, 17);
  LKV_CND(8, 16); LKV_CND(7, 11); LKV_CND(6, 10); LKV_CND(5, 9); LKV_CND(4, 8); LKV_CND(3, 3); LKV_CND(2, 2);
  LKV_CND(1, 1); LKV_CND(0, 0);
  return id;
}
#undef LKV_CMP
#undef LKV_CND

// One stage of the bf16 sweep.  `cur` holds stage st (its copy was waited
// for); the copy of stage st + kBf16Ring - 1 goes into `nxt`, the buffer that
// stage st - 1 used.
template <int kKT>
__device__ __forceinline__ void bf16_stage(const char* cur, char* nxt, const uint4* fslice,
                                           const float* cslice, int st, int n_stages, int wave, int lane, int h,
                                           const bf16x8_t (&b)[kKT][kBf16Steps], float (&best)[kKT],
                                           int (&bidx)[kKT]) {
  wait_vm_stages(min(kBf16Ring - 2, n_stages - 1 - st));
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();   // stage st is in LDS for all waves; stage st-1's buffer is free
  const bool copy_next = st + kBf16Ring - 1 < n_stages;
  const uint4* s_frag = reinterpret_cast<const uint4*>(cur);
  const float* s_cn = reinterpret_cast<const float*>(cur + kBf16StageTiles * kBf16TileU4 * 16);
  const int t0 = st * kBf16StageTiles;
#pragma unroll
  for (int tt = 0; tt < kBf16StageTiles; ++tt) {
    // spread the copy of stage st + kBf16Ring - 1 over the stage's tiles
    if (copy_next) {
      const int per = (kBf16DmaPerWave + kBf16StageTiles - 1) / kBf16StageTiles;
      stage_async_part(fslice, cslice, st + kBf16Ring - 1, nxt, wave, lane, tt * per,
                       min(kBf16DmaPerWave, (tt + 1) * per));
    }
    bf16x8_t a[kBf16Steps];
#pragma unroll
    for (int s = 0; s < kBf16Steps; ++s)
      a[s] = __builtin_bit_cast(bf16x8_t, s_frag[(tt * kBf16Steps + s) * 64 + lane]);
    floatx16 cn;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const float4 x = *reinterpret_cast<const float4*>(&s_cn[tt * kTileC + 8 * g + 4 * h]);
      cn[4 * g + 0] = x.x; cn[4 * g + 1] = x.y; cn[4 * g + 2] = x.z; cn[4 * g + 3] = x.w;
    }
    const int cbase = (t0 + tt) * kTileC + 4 * h;
    // independent accumulation chains (one per key tile), interleaved step by
    // step so consecutive MFMAs never wait on each other
    floatx16 acc[kKT];
#pragma unroll
    for (int kt = 0; kt < kKT; ++kt)
      acc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0], b[kt][0], cn, 0, 0, 0);
#pragma unroll
    for (int s = 1; s < kBf16Steps; ++s)
#pragma unroll
      for (int kt = 0; kt < kKT; ++kt)
        acc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s], b[kt][s], acc[kt], 0, 0, 0);
#pragma unroll
    for (int kt = 0; kt < kKT; ++kt) {
      const float m = tile_min(acc[kt]);
      const bool better = m < best[kt];
      // wave-uniform branch: EXEC stays all-ones, lanes select their update.
      // The predicate goes through an opaque register so the compiler cannot
      // turn the selects back into an EXEC-masked block.
      if (__builtin_amdgcn_ballot_w64(better)) {
        int sel = better ? 1 : 0;
        int id = cbase + tile_find(acc[kt], m);
        asm volatile("" : "+v"(sel), "+v"(id));
        bidx[kt] = sel ? id : bidx[kt];
        best[kt] = sel ? m : best[kt];
      }
    }
  }
}

// The whole sweep over the centroid stages.  The four ring buffers are
// restrict parameters of this one inlined function, so every asynchronous
// copy and every LDS read below carries alias scopes that tell the compiler
// which buffer it touches; it then waits only where the code says so instead
// of draining all copies in flight before each read.  best/bidx come in
// holding the starting bound (and -1).
template <int kKT>
__device__ __forceinline__ void bf16_sweep(char* __restrict__ r0, char* __restrict__ r1, char* __restrict__ r2,
                                           char* __restrict__ r3, const uint4* fslice, const float* cslice,
                                           int n_stages, int wave, int lane, int h,
                                           const bf16x8_t (&b)[kKT][kBf16Steps], float (&best)[kKT],
                                           int (&bidx)[kKT]) {
  // the first kBf16Ring - 1 stages were copied by the caller (bf16_prologue)
  for (int st = 0; st < n_stages; st += kBf16Ring) {
    bf16_stage<kKT>(r0, r3, fslice, cslice, st, n_stages, wave, lane, h, b, best, bidx);
    if (st + 1 >= n_stages) break;
    bf16_stage<kKT>(r1, r0, fslice, cslice, st + 1, n_stages, wave, lane, h, b, best, bidx);
    if (st + 2 >= n_stages) break;
    bf16_stage<kKT>(r2, r1, fslice, cslice, st + 2, n_stages, wave, lane, h, b, best, bidx);
    if (st + 3 >= n_stages) break;
    bf16_stage<kKT>(r3, r2, fslice, cslice, st + 3, n_stages, wave, lane, h, b, best, bidx);
  }
}

// Copies of the first kBf16Ring - 1 stages, issued before anything else the
// block loads, so their latency overlaps the key loads and the bound.
__device__ __forceinline__ void bf16_prologue(char* __restrict__ r0, char* __restrict__ r1, char* __restrict__ r2,
                                              const uint4* fslice, const float* cslice, int n_stages, int wave,
                                              int lane) {
  stage_async(fslice, cslice, 0, r0, wave, lane);
  if (n_stages > 1) stage_async(fslice, cslice, 1, r1, wave, lane);
  if (n_stages > 2) stage_async(fslice, cslice, 2, r2, wave, lane);
}

// bf16 keys: each wave holds kBf16KeyTiles tiles of 32 keys as MFMA B operands
// for the whole sweep; centroid tiles stream through a ring of kBf16Ring LDS
// stage buffers, copied kBf16Ring - 1 stages ahead.  Lane l owns key column
// l % 32 and rows 8*(v/4) + 4*(l/32) + (v%4) of each 32x32 result, so the
// argmin over a tile is in-lane; the two lane halves merge at the end.
__global__ __launch_bounds__(kBf16Threads, 8 / kBf16Waves)
void assign_bf16_kernel(const uint16_t* __restrict__ keys, const uint4* __restrict__ frag,
                        const float* __restrict__ cnorm, int32_t* __restrict__ assign,
                        int32_t* __restrict__ counts, int n_tokens, int n_clusters, int n_ctiles,
                        int blocks_per_slice, int hist_in_lds, int use_bound, uint4* __restrict__ kswz,
                        int kswz_mode, int32_t* __restrict__ dirty) {
  __shared__ __align__(16) char s_ring0[kBf16StageBytes];
  __shared__ __align__(16) char s_ring1[kBf16StageBytes];
  __shared__ __align__(16) char s_ring2[kBf16StageBytes];
  __shared__ __align__(16) char s_ring3[kBf16StageBytes];
  static_assert(kBf16Ring == 4, "the stage loop below is unrolled for four buffers");

  const int lb = xcd_local_block(blockIdx.x, gridDim.x);
  const int slice = lb / blocks_per_slice;
  const int kb = lb - slice * blocks_per_slice;
  // the wave index lives in an SGPR (it addresses the copies every stage)
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, h = lane >> 5,
            j = lane & 31;
  const int key_base = kb * kBf16KeysPerBlock + wave * (32 * kBf16KeyTiles);
  const uint16_t* kslice = keys + (size_t)slice * n_tokens * kHeadDim;
  const uint4* fslice = frag + (size_t)slice * n_ctiles * kBf16TileU4;
  const float* cslice = cnorm + (size_t)slice * n_ctiles * kTileC;
  const int n_stages = n_ctiles / kBf16StageTiles;   // n_ctiles is padded to whole stages

  // Start-up latency is the block's fixed cost, so the loads that do not
  // depend on each other are issued together: the ring's first copies, the
  // previous assignment (for the bound), then the keys.
  bf16_prologue(s_ring0, s_ring1, s_ring2, fslice, cslice, n_stages, wave, lane);
  int zp[kBf16KeyTiles];
#pragma unroll
  for (int kt = 0; kt < kBf16KeyTiles; ++kt) {
    const int key = key_base + kt * 32 + j;
    zp[kt] = (use_bound && key < n_tokens) ? assign[(size_t)slice * n_tokens + key] : -1;
  }
  // Key operands.  In B-operand order a load instruction touches 64 rows
  // (16 bytes of each), which makes the block's start slow; so the first
  // iteration of a prefill also stores the operands in that order (kswz_mode
  // 1, one contiguous KiB per instruction, padding keys zero), and the later
  // iterations read them back contiguously (kswz_mode 2).
  bf16x8_t b[kBf16KeyTiles][kBf16Steps];
  uint4* zs = kswz + (((size_t)slice * blocks_per_slice + kb) * kBf16Waves + wave) * (kBf16KeyTiles * kBf16Steps * 64);
  if (kswz_mode == 2) {
#pragma unroll
    for (int kt = 0; kt < kBf16KeyTiles; ++kt)
#pragma unroll
      for (int s = 0; s < kBf16Steps; ++s) b[kt][s] = __builtin_bit_cast(bf16x8_t, zs[(kt * kBf16Steps + s) * 64 + lane]);
  } else {
#pragma unroll
    for (int kt = 0; kt < kBf16KeyTiles; ++kt) {
      const int key = key_base + kt * 32 + j;
      const uint4* src = reinterpret_cast<const uint4*>(kslice + (size_t)key * kHeadDim + 64 * h);
#pragma unroll
      for (int s = 0; s < kBf16Steps; ++s) {
        uint4 v = key < n_tokens ? src[s] : make_uint4(0, 0, 0, 0);
        b[kt][s] = __builtin_bit_cast(bf16x8_t, v);
      }
    }
    if (kswz_mode == 1) {
#pragma unroll
      for (int kt = 0; kt < kBf16KeyTiles; ++kt)
#pragma unroll
        for (int s = 0; s < kBf16Steps; ++s) zs[(kt * kBf16Steps + s) * 64 + lane] = __builtin_bit_cast(uint4, b[kt][s]);
    }
  }
  // Starting bound.  From the second Lloyd iteration on, assign holds the
  // previous assignment; the key's distance to that centroid (computed on the
  // VALU over the same bf16 operands) plus a margin is an upper bound on the
  // matrix-core value of its nearest centroid: both evaluations of D differ
  // from the exact value by at most ~60 x 2^-24 x (||c||^2 + 2 sum|c_i k_i|)
  // <= 7.2e-6 (||c||^2 + ||k||^2), and the margin is 3e-5 of that.  Tiles whose
  // minimum does not beat the bound skip the index search; the nearest
  // centroid's value is strictly below it, so the result is unchanged.
  float best[kBf16KeyTiles];
  int bidx[kBf16KeyTiles];
#pragma unroll
  for (int kt = 0; kt < kBf16KeyTiles; ++kt) {
    bidx[kt] = -1;
    best[kt] = __builtin_inff();
    const bool have = zp[kt] >= 0 && zp[kt] < n_clusters;
    if (__builtin_amdgcn_ballot_w64(have)) {
      typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
      const int zc = have ? zp[kt] : 0;
      // the lane's 64 dimensions of -2 op(c): A-fragment row zc % 32, half h
      const uint4* f = fslice + (size_t)(zc / kTileC) * kBf16TileU4 + (zc % kTileC) + 32 * h;
      float p = 0.f, kk = 0.f;
#pragma unroll
      for (int s = 0; s < kBf16Steps; ++s) {
        const uint4 fa = f[s * 64];
        const uint4 kv = __builtin_bit_cast(uint4, b[kt][s]);
        const uint32_t fw[4] = {fa.x, fa.y, fa.z, fa.w};
        const uint32_t kw[4] = {kv.x, kv.y, kv.z, kv.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const bf16x2_t kq = __builtin_bit_cast(bf16x2_t, kw[q]);
          p = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, fw[q]), kq, p, false);
          kk = __builtin_amdgcn_fdot2_f32_bf16(kq, kq, kk, false);
        }
      }
      p += __shfl_xor(p, 32, kWave);
      kk += __shfl_xor(kk, 32, kWave);
      const float cn = cslice[zc];
      const float u = cn + p + 3e-5f * (cn + kk);
      if (have && u < __builtin_inff()) best[kt] = u;   // false for NaN
    }
  }
  // the key operands are complete before the sweep starts, so no key load is
  // pending inside the stage loop (the loop then only waits for its copies);
  // the compiler does not read that wait, so every key register is also used
  // here, which makes it complete the loads before the loop, not inside it
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
  for (int kt = 0; kt < kBf16KeyTiles; ++kt)
#pragma unroll
    for (int s = 0; s < kBf16Steps; ++s) asm volatile("" ::"v"(b[kt][s]));
  bf16_sweep<kBf16KeyTiles>(s_ring0, s_ring1, s_ring2, s_ring3, fslice, cslice, n_stages, wave, lane, h, b, best,
                            bidx);

  int zi[kBf16KeyTiles];
  bool zv[kBf16KeyTiles];
#pragma unroll
  for (int kt = 0; kt < kBf16KeyTiles; ++kt) {
    const float ob = __shfl_xor(best[kt], 32, kWave);
    const int oi = __shfl_xor(bidx[kt], 32, kWave);
    // a half with no value below its starting bound holds index -1
    if (bidx[kt] < 0 || (oi >= 0 && (ob < best[kt] || (ob == best[kt] && oi < bidx[kt])))) {
      best[kt] = ob;
      bidx[kt] = oi;
    }
    if (bidx[kt] < 0) bidx[kt] = 0;   // only reachable with non-finite inputs
    const int key = key_base + kt * 32 + j;
    zi[kt] = bidx[kt];
    zv[kt] = (h == 0) && key < n_tokens;
    if (zv[kt]) assign[(size_t)slice * n_tokens + key] = bidx[kt];
    // a key that changed cluster marks both clusters for the update
    if (dirty && zv[kt] && bidx[kt] != zp[kt]) {
      dirty[(size_t)slice * n_clusters + bidx[kt]] = 1;
      if (zp[kt] >= 0 && zp[kt] < n_clusters) dirty[(size_t)slice * n_clusters + zp[kt]] = 1;
    }
  }
  if (counts) {
    __syncthreads();
    block_histogram(reinterpret_cast<int*>(s_ring0), hist_in_lds, n_clusters,
                    counts + (size_t)slice * n_clusters, zi, zv, kBf16KeyTiles);
  }
}

// fp32 keys: the same scheme with 32x32x2 fp32 MFMAs (64 steps per dot product)
// and one 32-key tile per wave.
__global__ __launch_bounds__(kAssignThreads, 2)
void assign_f32_kernel(const float* __restrict__ keys, const uint4* __restrict__ frag,
                       const float* __restrict__ cnorm, int32_t* __restrict__ assign,
                       int32_t* __restrict__ counts, int n_tokens, int n_clusters, int n_ctiles,
                       int blocks_per_slice, int hist_in_lds) {
  extern __shared__ __align__(16) char smem[];
  uint4* s_frag = reinterpret_cast<uint4*>(smem);
  float* s_cn = reinterpret_cast<float*>(smem + kF32StageTiles * kF32TileU4 * 16);

  const int slice = blockIdx.x / blocks_per_slice;
  const int kb = blockIdx.x - slice * blocks_per_slice;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, h = lane >> 5, j = lane & 31;
  const int key = kb * kF32KeysPerBlock + wave * 32 + j;
  const float* kslice = keys + (size_t)slice * n_tokens * kHeadDim;

  float b[64];
  {
    const float4* src = reinterpret_cast<const float4*>(kslice + (size_t)key * kHeadDim + 64 * h);
#pragma unroll
    for (int s4 = 0; s4 < 16; ++s4) {
      float4 v = key < n_tokens ? src[s4] : make_float4(0.f, 0.f, 0.f, 0.f);
      b[4 * s4 + 0] = v.x; b[4 * s4 + 1] = v.y; b[4 * s4 + 2] = v.z; b[4 * s4 + 3] = v.w;
    }
  }
  float best = __builtin_inff();
  int bidx = 0;
  const uint4* fslice = frag + (size_t)slice * n_ctiles * kF32TileU4;
  const float* cslice = cnorm + (size_t)slice * n_ctiles * kTileC;
  for (int t0 = 0; t0 < n_ctiles; t0 += kF32StageTiles) {
    const int nt = min(kF32StageTiles, n_ctiles - t0);
    __syncthreads();
    for (int i = tid; i < nt * kF32TileU4; i += kAssignThreads) s_frag[i] = fslice[(size_t)t0 * kF32TileU4 + i];
    for (int i = tid; i < nt * kTileC; i += kAssignThreads) s_cn[i] = cslice[t0 * kTileC + i];
    __syncthreads();
    for (int tt = 0; tt < nt; ++tt) {
      floatx16 acc;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const float4 x = *reinterpret_cast<const float4*>(&s_cn[tt * kTileC + 8 * g + 4 * h]);
        acc[4 * g + 0] = x.x; acc[4 * g + 1] = x.y; acc[4 * g + 2] = x.z; acc[4 * g + 3] = x.w;
      }
#pragma unroll
      for (int s4 = 0; s4 < 16; ++s4) {
        const float4 a4 = __builtin_bit_cast(float4, s_frag[(tt * 16 + s4) * 64 + lane]);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4.x, b[4 * s4 + 0], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4.y, b[4 * s4 + 1], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4.z, b[4 * s4 + 2], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4.w, b[4 * s4 + 3], acc, 0, 0, 0);
      }
      const int cbase = (t0 + tt) * kTileC + 4 * h;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float x = acc[v];
        const int c = cbase + 8 * (v >> 2) + (v & 3);
        if (x < best) { best = x; bidx = c; }
      }
    }
  }
  const float ob = __shfl_xor(best, 32, kWave);
  const int oi = __shfl_xor(bidx, 32, kWave);
  if (ob < best || (ob == best && oi < bidx)) { best = ob; bidx = oi; }
  const bool valid = (h == 0) && key < n_tokens;
  if (valid) assign[(size_t)slice * n_tokens + key] = bidx;
  if (counts) {
    __syncthreads();
    int zi[1] = {bidx};
    bool zv[1] = {valid};
    block_histogram(reinterpret_cast<int*>(smem), hist_in_lds, n_clusters,
                    counts + (size_t)slice * n_clusters, zi, zv, 1);
  }
}

constexpr int kCountKeys = 1024;

// counts[s][c] = number of keys with assign == c (used by the standalone update).
__global__ void count_kernel(const int32_t* __restrict__ assign, int32_t* __restrict__ counts, int n_tokens,
                             int n_clusters, int blocks_per_slice, int hist_in_lds) {
  extern __shared__ __align__(16) char smem[];
  const int slice = blockIdx.x / blocks_per_slice;
  const int kb = blockIdx.x - slice * blocks_per_slice;
  int zi[4];
  bool zv[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int i = kb * kCountKeys + q * 256 + threadIdx.x;
    zv[q] = i < n_tokens;
    zi[q] = zv[q] ? assign[(size_t)slice * n_tokens + i] : 0;
    zv[q] = zv[q] && zi[q] >= 0 && zi[q] < n_clusters;
  }
  block_histogram(reinterpret_cast<int*>(smem), hist_in_lds, n_clusters,
                  counts + (size_t)slice * n_clusters, zi, zv, 4);
}

// Per slice: offsets[c] = sum of counts[<c], offsets[C] = total; cursor = offsets.
__global__ __launch_bounds__(1024)
void scan_kernel(const int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
                 int32_t* __restrict__ cursor, int n_clusters) {
  __shared__ int s_warp[16];
  __shared__ int s_carry;
  const int slice = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int32_t* cnt = counts + (size_t)slice * n_clusters;
  int32_t* off = offsets + (size_t)slice * (n_clusters + 1);
  int32_t* cur = cursor + (size_t)slice * n_clusters;
  if (tid == 0) s_carry = 0;
  __syncthreads();
  for (int base = 0; base < n_clusters; base += 1024) {
    const int c = base + tid;
    const int v = c < n_clusters ? cnt[c] : 0;
    int x = v;  // inclusive wave scan
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o, kWave);
      if (lane >= o) x += y;
    }
    if (lane == 63) s_warp[w] = x;
    __syncthreads();
    int wprefix = 0;
    for (int q = 0; q < w; ++q) wprefix += s_warp[q];
    const int carry = s_carry;
    const int excl = carry + wprefix + x - v;
    if (c < n_clusters) {
      off[c] = excl;
      cur[c] = excl;
    }
    __syncthreads();
    if (tid == 1023) s_carry = excl + v;
    __syncthreads();
  }
  if (tid == 0) off[n_clusters] = s_carry;
}

constexpr int kScatterKeys = 1024;

// members[s][offsets[z] + k] = i for the keys i of each cluster z, k unique per key.
__global__ void scatter_kernel(const int32_t* __restrict__ assign, int32_t* __restrict__ cursor,
                               int32_t* __restrict__ members, int n_tokens, int n_clusters,
                               int blocks_per_slice, int lds_ok) {
  extern __shared__ __align__(16) char smem[];
  int* hist = reinterpret_cast<int*>(smem);
  int* base = hist + n_clusters;
  const int slice = blockIdx.x / blocks_per_slice;
  const int kb = blockIdx.x - slice * blocks_per_slice;
  const int tid = threadIdx.x;
  int32_t* cur = cursor + (size_t)slice * n_clusters;
  int32_t* mem = members + (size_t)slice * n_tokens;
  int z[4], pos[4];
  bool ok[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int i = kb * kScatterKeys + q * 256 + tid;
    ok[q] = i < n_tokens;
    z[q] = ok[q] ? assign[(size_t)slice * n_tokens + i] : 0;
    ok[q] = ok[q] && z[q] >= 0 && z[q] < n_clusters;   // same keys as the count
    if (!ok[q]) z[q] = 0;
  }
  if (!lds_ok) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (ok[q]) mem[atomicAdd(&cur[z[q]], 1)] = kb * kScatterKeys + q * 256 + tid;
    return;
  }
  for (int i = tid; i < n_clusters; i += 256) hist[i] = 0;
  __syncthreads();
#pragma unroll
  for (int q = 0; q < 4; ++q) pos[q] = ok[q] ? atomicAdd(&hist[z[q]], 1) : 0;
  __syncthreads();
  for (int i = tid; i < n_clusters; i += 256)
    if (hist[i]) base[i] = atomicAdd(&cur[i], hist[i]);
  __syncthreads();
#pragma unroll
  for (int q = 0; q < 4; ++q)
    if (ok[q]) mem[base[z[q]] + pos[q]] = kb * kScatterKeys + q * 256 + tid;
}

// One wave per (slice, cluster): mean of the member keys, float64 sum.
// A key row is read as 16-byte pieces: kLpr lanes per row, so one wave load
// covers kRpl rows and four loads are in flight; each lane accumulates its
// dims in float64 and the row groups are summed across lanes at the end.
// With frag given, the wave also writes the next iteration's matrix operand
// for this centroid (-2 op(c) in A-fragment order, and ||op(c)||^2), the work
// prep_operand_kernel does for the first iteration; with zero_counts it
// clears the cluster's count for the next assignment.
template <class T>
__global__ void centroid_update_kernel(const T* __restrict__ keys, const int32_t* __restrict__ members,
                                       const int32_t* __restrict__ offsets, int32_t* __restrict__ counts,
                                       const float* centroids_in, float* centroids_out, int stride, int n_tokens,
                                       int n_clusters, int64_t n_rows, uint4* __restrict__ frag,
                                       float* __restrict__ cnorm, int n_ctiles, int zero_counts,
                                       int32_t* __restrict__ dirty, int skip_clean) {
  constexpr int kDims = 16 / sizeof(T);          // dims per 16-byte piece (8 bf16, 4 fp32)
  constexpr int kLpr = kHeadDim / kDims;         // lanes per row
  constexpr int kRpl = kWave / kLpr;             // rows per wave load
  constexpr int kUnroll = 4;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n_rows) return;
  const int lane = threadIdx.x & 63;
  const int64_t s = row / n_clusters;
  const int c = (int)(row - s * n_clusters);
  const int n = counts[s * n_clusters + c];
  float* dst = centroids_out + ((size_t)s * stride + c) * kHeadDim;
  if (dirty) {
    // a cluster that no key entered or left keeps its members, hence its
    // mean and the operand prepared from it; the flag is cleared for the
    // next assignment either way
    const int was_dirty = dirty[row];
    if (lane == 0) dirty[row] = 0;
    if (skip_clean && !was_dirty) {
      if (zero_counts && lane == 0) counts[s * n_clusters + c] = 0;
      return;
    }
  }
  if (n == 0) {
    // empty: the centroid (and its operand from the previous preparation) stay
    if (centroids_in != centroids_out) {
      const float* src = centroids_in + ((size_t)s * stride + c) * kHeadDim;
      dst[2 * lane] = src[2 * lane];
      dst[2 * lane + 1] = src[2 * lane + 1];
    }
    return;
  }
  const int off = offsets[s * (n_clusters + 1) + c];
  const int32_t* mem = members + (size_t)s * n_tokens + off;
  const T* kslice = keys + (size_t)s * n_tokens * kHeadDim;
  const int sub = lane % kLpr, grp = lane / kLpr;
  double acc[kDims];
#pragma unroll
  for (int e = 0; e < kDims; ++e) acc[e] = 0.0;
  for (int m0 = 0; m0 < n; m0 += kWave) {
    const int mine = (m0 + lane < n) ? mem[m0 + lane] : 0;
    const int cnt = min(kWave, n - m0);
    for (int q = 0; q < cnt; q += kRpl * kUnroll) {
      uint4 x[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int r = q + u * kRpl + grp;
        const int tok = __shfl(mine, r & (kWave - 1), kWave);
        x[u] = r < cnt ? reinterpret_cast<const uint4*>(kslice + (size_t)tok * kHeadDim)[sub]
                       : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const T* v = reinterpret_cast<const T*>(&x[u]);
#pragma unroll
        for (int e = 0; e < kDims; ++e) acc[e] += (double)load_as_f32(v, e);
      }
    }
  }
#pragma unroll
  for (int o = kLpr; o < kWave; o <<= 1)
#pragma unroll
    for (int e = 0; e < kDims; ++e) acc[e] += __shfl_xor(acc[e], o, kWave);
  if (grp != 0) return;
  // lanes 0..kLpr-1 hold dims kDims*lane ..
  float mean[kDims];
#pragma unroll
  for (int e = 0; e < kDims; ++e) mean[e] = (float)(acc[e] / (double)n);
  float4* d4 = reinterpret_cast<float4*>(dst + kDims * sub);
#pragma unroll
  for (int e = 0; e < kDims; e += 4) d4[e / 4] = make_float4(mean[e], mean[e + 1], mean[e + 2], mean[e + 3]);
  if (zero_counts && sub == 0) counts[s * n_clusters + c] = 0;
  if (!frag) return;
  // next iteration's operand: same layout and values as prep_operand_kernel
  const int t = c / kTileC, ci = c % kTileC;
  const int d0 = kDims * sub, hh = d0 >> 6;
  const int flane = hh * 32 + ci;
  double nrm = 0.0;
  if (sizeof(T) == 2) {
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      const float o0 = bf16_to_f32(f32_to_bf16(mean[e])), o1 = bf16_to_f32(f32_to_bf16(mean[e + 1]));
      nrm += (double)o0 * o0 + (double)o1 * o1;
      w[e / 2] = (uint32_t)f32_to_bf16(-2.f * o0) | ((uint32_t)f32_to_bf16(-2.f * o1) << 16);
    }
    const int step = (d0 & 63) >> 3;
    frag[((size_t)s * n_ctiles + t) * kBf16TileU4 + step * 64 + flane] = make_uint4(w[0], w[1], w[2], w[3]);
  } else {
#pragma unroll
    for (int e = 0; e < kDims; ++e) nrm += (double)mean[e] * mean[e];
    const int step = d0 & 63;   // 4 consecutive steps, one float4 of the fp32 layout
    float* f = reinterpret_cast<float*>(frag + ((size_t)s * n_ctiles + t) * kF32TileU4);
    *reinterpret_cast<float4*>(f + ((size_t)(step >> 2) * 64 + flane) * 4) =
        make_float4(-2.f * mean[0], -2.f * mean[1], -2.f * mean[2], -2.f * mean[3]);
  }
#pragma unroll
  for (int o = 1; o < kLpr; o <<= 1) nrm += __shfl_xor(nrm, o, kWave);
  if (sub == 0) cnorm[(size_t)s * n_ctiles * kTileC + c] = (float)nrm;
}

// One wave per (slice, cluster): member ids sorted ascending into perm (rank =
// number of smaller ids, ids are distinct), and the unit-table entry.
__global__ void finalize_kernel(const int32_t* __restrict__ members, const int32_t* __restrict__ offsets,
                                const int32_t* __restrict__ counts, int32_t* __restrict__ perm,
                                int32_t* __restrict__ unit_start, int32_t* __restrict__ unit_size,
                                int units_cap, int n_tokens, int n_clusters, int64_t n_rows) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n_rows) return;
  const int lane = threadIdx.x & 63;
  const int64_t s = row / n_clusters;
  const int c = (int)(row - s * n_clusters);
  const int n = counts[s * n_clusters + c];
  const int off = offsets[s * (n_clusters + 1) + c];
  if (lane == 0) {
    unit_start[s * units_cap + c] = off;
    unit_size[s * units_cap + c] = n;
  }
  const int32_t* mem = members + (size_t)s * n_tokens + off;
  int32_t* out = perm + (size_t)s * n_tokens + off;
  if (n <= 64) {
    const int mine = lane < n ? mem[lane] : 0x7fffffff;
    int rank = 0;
    for (int q = 0; q < n; ++q) rank += __shfl(mine, q, kWave) < mine;
    if (lane < n) out[rank] = mine;
    return;
  }
  for (int i = lane; i < n; i += 64) {
    const int mine = mem[i];
    int rank = 0;
    for (int q = 0; q < n; ++q) rank += mem[q] < mine;
    out[rank] = mine;
  }
}

// pool[s][r] = src[s][perm[s][r]] for r < n_tokens; 16 lanes per row.
template <class T>
__global__ void pack_pool_kernel(const T* __restrict__ src, const int32_t* __restrict__ perm,
                                 T* __restrict__ pool, int64_t pool_rows, int n_tokens, int64_t n_rows) {
  // 16 rows per block of 256 per round; a grid smaller than n_rows / 16
  // blocks strides over the rest (a pack that shares the chip with clustering)
  const int sub = threadIdx.x & 15;
  for (int64_t g = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4); g < n_rows; g += (int64_t)gridDim.x * 16) {
    const int64_t s = g / n_tokens;
    const int r = (int)(g - s * n_tokens);
    const int tok = min(max(perm[s * n_tokens + r], 0), n_tokens - 1);   // perm may come from the caller
    constexpr int kU4 = kHeadDim * sizeof(T) / 16;
    const uint4* a = reinterpret_cast<const uint4*>(src + ((size_t)s * n_tokens + tok) * kHeadDim);
    uint4* b = reinterpret_cast<uint4*>(pool + ((size_t)s * pool_rows + r) * kHeadDim);
#pragma unroll
    for (int q = sub; q < kU4; q += 16) b[q] = a[q];
  }
}

__global__ void fill_i32_kernel(int32_t* __restrict__ p, int32_t v, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// Page-level index: one wave per (slice, page).  Lane l sums dims 2l, 2l+1 of
// the page's keys in float64 (row order) and writes their mean rounded once
// to float32; the page's K/V rows are copied to the pool in token order.
template <class T>
__global__ __launch_bounds__(256)
void page_units_kernel(const T* __restrict__ keys, const T* __restrict__ values, int n_tokens, int page_len,
                       int n_pages, int64_t n_items, float* __restrict__ reps, int units_cap,
                       int32_t* __restrict__ unit_start, int32_t* __restrict__ unit_size, T* __restrict__ k_pool,
                       T* __restrict__ v_pool, int64_t pool_rows) {
  const int64_t item = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (item >= n_items) return;
  const int lane = threadIdx.x & 63;
  const int64_t s = item / n_pages;
  const int p = (int)(item - s * n_pages);
  const int a = p * page_len;
  const int len = min(page_len, n_tokens - a);
  double x0 = 0.0, x1 = 0.0;
  for (int r = 0; r < len; ++r) {
    const size_t o = ((size_t)s * n_tokens + a + r) * kHeadDim + 2 * lane;
    x0 += (double)load_as_f32(keys, o);
    x1 += (double)load_as_f32(keys, o + 1);
    if (k_pool) {
      const size_t po = ((size_t)s * pool_rows + a + r) * kHeadDim + 2 * lane;
      k_pool[po] = keys[o];
      k_pool[po + 1] = keys[o + 1];
      if (v_pool) {
        v_pool[po] = values[o];
        v_pool[po + 1] = values[o + 1];
      }
    }
  }
  float* rep = reps + ((size_t)s * units_cap + p) * kHeadDim;
  rep[2 * lane] = (float)(x0 / (double)len);
  rep[2 * lane + 1] = (float)(x1 / (double)len);
  if (lane == 0) {
    unit_start[s * units_cap + p] = a;
    unit_size[s * units_cap + p] = len;
  }
}

// ------------------------------------------------------------------ host side

struct Ws {
  uint4* frag;
  float* cnorm;
  int32_t* counts;
  int32_t* offsets;
  int32_t* cursor;
  int32_t* members;
  int32_t* dirty;   // per cluster: a key entered or left it in the last assignment
  uint4* kswz;   // bf16 key operands in B-operand order (kswz_mode of the assignment)
  size_t bytes;
};

// Centroid tiles per slice; bf16 pads to whole LDS stages (padding rows have a
// zero operand and an infinite norm, so they never win).
int n_ctiles_for(int n_clusters, int dtype) {
  const int t = ceil_div(n_clusters, kTileC);
  return dtype == LOUISKV_BF16 ? ceil_div(t, kBf16StageTiles) * kBf16StageTiles : t;
}

Ws carve(void* base, int64_t n_slices, int n_tokens, int n_clusters, int dtype) {
  Carver cv(base);
  const int n_ctiles = n_ctiles_for(n_clusters, dtype);
  const int tile_u4 = dtype == LOUISKV_BF16 ? kBf16TileU4 : kF32TileU4;
  Ws w;
  w.frag = cv.take<uint4>((size_t)n_slices * n_ctiles * tile_u4);
  w.cnorm = cv.take<float>((size_t)n_slices * n_ctiles * kTileC);
  w.counts = cv.take<int32_t>((size_t)n_slices * n_clusters);
  w.offsets = cv.take<int32_t>((size_t)n_slices * (n_clusters + 1));
  w.cursor = cv.take<int32_t>((size_t)n_slices * n_clusters);
  w.members = cv.take<int32_t>((size_t)n_slices * n_tokens);
  w.dirty = cv.take<int32_t>((size_t)n_slices * n_clusters);
  w.kswz = dtype == LOUISKV_BF16
               ? cv.take<uint4>((size_t)n_slices * ceil_div(n_tokens, kBf16KeysPerBlock) * kBf16KeysPerBlock * 16)
               : nullptr;
  w.bytes = align_up(cv.used, 256);
  return w;
}

constexpr size_t kMaxHistLds = 64 * 1024;

int launch_prep(const float* reps, int stride, int64_t S, int C, int dtype, const Ws& w, bool zero_counts,
                hipStream_t st) {
  const int n_ctiles = n_ctiles_for(C, dtype);
  const int64_t rows = S * n_ctiles * kTileC;
  const int grid = (int)((rows + 3) / 4);
  if (dtype == LOUISKV_BF16)
    prep_operand_kernel<true><<<grid, 256, 0, st>>>(reps, stride, C, n_ctiles, w.frag, w.cnorm,
                                                     zero_counts ? w.counts : nullptr, rows);
  else
    prep_operand_kernel<false><<<grid, 256, 0, st>>>(reps, stride, C, n_ctiles, w.frag, w.cnorm,
                                                      zero_counts ? w.counts : nullptr, rows);
  LKV_CHECK_LAUNCH();
  return LOUISKV_OK;
}

// use_bound: assign holds a valid previous assignment; kswz_mode: 0 keys only,
// 1 keys and store the operand copy, 2 read the copy (bf16 path only).
// mark_dirty: flag the clusters a key enters or leaves (bf16 path; needs the
// previous assignment, i.e. use_bound).
int launch_assign(const void* keys, int dtype, int64_t S, int N, int C, const Ws& w, int32_t* assign,
                  bool with_counts, bool use_bound, int kswz_mode, hipStream_t st, bool mark_dirty = false) {
  const int n_ctiles = n_ctiles_for(C, dtype);
  if (dtype == LOUISKV_BF16) {
    const int bps = ceil_div(N, kBf16KeysPerBlock);
    const bool hist_lds = (size_t)C * 4 <= (size_t)kBf16StageBytes;
    assign_bf16_kernel<<<(unsigned)(S * bps), kBf16Threads, 0, st>>>(
        static_cast<const uint16_t*>(keys), w.frag, w.cnorm, assign, with_counts ? w.counts : nullptr, N, C,
        n_ctiles, bps, hist_lds ? 1 : 0, use_bound ? 1 : 0, w.kswz, kswz_mode,
        mark_dirty && use_bound ? w.dirty : nullptr);
  } else {
    const int bps = ceil_div(N, kF32KeysPerBlock);
    size_t lds = (size_t)kF32StageTiles * (kF32TileU4 * 16 + kTileC * 4);
    const bool hist_lds = (size_t)C * 4 <= std::max(lds, kMaxHistLds);
    if (with_counts && hist_lds) lds = std::max(lds, (size_t)C * 4);
    assign_f32_kernel<<<(unsigned)(S * bps), kAssignThreads, lds, st>>>(
        static_cast<const float*>(keys), w.frag, w.cnorm, assign, with_counts ? w.counts : nullptr, N, C,
        n_ctiles, bps, hist_lds ? 1 : 0);
  }
  LKV_CHECK_LAUNCH();
  return LOUISKV_OK;
}

int launch_scan_scatter(const int32_t* assign, int64_t S, int N, int C, const Ws& w, hipStream_t st) {
  scan_kernel<<<(unsigned)S, 1024, 0, st>>>(w.counts, w.offsets, w.cursor, C);
  LKV_CHECK_LAUNCH();
  const int bps = ceil_div(N, kScatterKeys);
  const bool lds_ok = (size_t)C * 8 <= kMaxHistLds;
  scatter_kernel<<<(unsigned)(S * bps), 256, lds_ok ? (size_t)C * 8 : 0, st>>>(assign, w.cursor, w.members, N, C,
                                                                              bps, lds_ok ? 1 : 0);
  LKV_CHECK_LAUNCH();
  return LOUISKV_OK;
}

// Centroid update; with prep_next, also the next iteration's operand and
// cleared counts (the work of launch_prep for the iterations after the first).
// dirty_mode: 0 no flags (every cluster), 1 every cluster and clear the
// flags, 2 only the flagged clusters (the others keep centroid and operand)
// and clear the flags.
int launch_sum(const void* keys, int dtype, int64_t S, int N, int C, const Ws& w, const float* cin, float* cout,
               int stride, bool prep_next, hipStream_t st, int dirty_mode = 0) {
  const int64_t rows = S * C;
  const int grid = (int)((rows + 3) / 4);
  const int n_ctiles = n_ctiles_for(C, dtype);
  uint4* frag = prep_next ? w.frag : nullptr;
  int32_t* dirty = dirty_mode ? w.dirty : nullptr;
  const int skip = dirty_mode == 2 ? 1 : 0;
  if (dtype == LOUISKV_BF16)
    centroid_update_kernel<uint16_t><<<grid, 256, 0, st>>>(static_cast<const uint16_t*>(keys), w.members,
                                                            w.offsets, w.counts, cin, cout, stride, N, C, rows, frag,
                                                            w.cnorm, n_ctiles, prep_next ? 1 : 0, dirty, skip);
  else
    centroid_update_kernel<float><<<grid, 256, 0, st>>>(static_cast<const float*>(keys), w.members, w.offsets,
                                                         w.counts, cin, cout, stride, N, C, rows, frag, w.cnorm,
                                                         n_ctiles, prep_next ? 1 : 0, dirty, skip);
  LKV_CHECK_LAUNCH();
  return LOUISKV_OK;
}

// Prompt K/V rows in perm order into the pools (each cluster one contiguous run).
int launch_pack(const void* keys, const void* values, int dtype, int64_t S, int N, const int32_t* perm, void* k_pool,
                void* v_pool, int64_t pool_rows, hipStream_t s, int max_grid = 0) {
  const int64_t prow = S * N;
  int pgrid = (int)((prow + 15) / 16);
  if (max_grid > 0) pgrid = std::min(pgrid, max_grid);
  for (int which = 0; which < 2; ++which) {
    void* pool = which == 0 ? k_pool : v_pool;
    const void* src = which == 0 ? keys : values;
    if (!pool) continue;
    if (dtype == LOUISKV_BF16)
      pack_pool_kernel<uint16_t><<<pgrid, 256, 0, s>>>(static_cast<const uint16_t*>(src), perm,
                                                        static_cast<uint16_t*>(pool), pool_rows, N, prow);
    else
      pack_pool_kernel<float><<<pgrid, 256, 0, s>>>(static_cast<const float*>(src), perm, static_cast<float*>(pool),
                                                     pool_rows, N, prow);
    LKV_CHECK_LAUNCH();
  }
  return LOUISKV_OK;
}


// Initial centroids, n_iters Lloyd iterations and the CSR/perm outputs, for
// arguments already validated (no pool write).
int run_cluster(const void* keys, int dtype, int64_t S, int N, int C, int n_iters, const int32_t* init_idx,
                float* reps, int units_cap, int32_t* unit_start, int32_t* unit_size, int32_t* assign, int32_t* perm,
                void* const* iter_events, const Ws& w, hipStream_t s) {
  int st;
  {
    const int64_t rows = S * C;
    const int grid = (int)((rows + 3) / 4);
    if (dtype == LOUISKV_BF16)
      init_centroids_kernel<uint16_t><<<grid, 256, 0, s>>>(static_cast<const uint16_t*>(keys), init_idx, reps,
                                                            N, C, units_cap, rows);
    else
      init_centroids_kernel<float><<<grid, 256, 0, s>>>(static_cast<const float*>(keys), init_idx, reps, N,
                                                         C, units_cap, rows);
    LKV_CHECK_LAUNCH();
  }
  // the first operand comes from the initial centroids; after that each
  // update writes the next one (and clears the counts) as it goes
  if ((st = launch_prep(reps, units_cap, S, C, dtype, w, true, s))) return st;
  for (int it = 0; it < n_iters; ++it) {
    if (iter_events) LKV_CHECK_HIP(hipEventRecord(reinterpret_cast<hipEvent_t>(iter_events[2 * it]), s));
    // from the second iteration on (bf16), the assignment flags the clusters
    // that keys entered or left and the update recomputes only those
    const bool track = dtype == LOUISKV_BF16;
    if ((st = launch_assign(keys, dtype, S, N, C, w, assign, true, it > 0, it == 0 ? 1 : 2, s, track)))
      return st;
    if (iter_events) LKV_CHECK_HIP(hipEventRecord(reinterpret_cast<hipEvent_t>(iter_events[2 * it + 1]), s));
    if ((st = launch_scan_scatter(assign, S, N, C, w, s))) return st;
    if ((st = launch_sum(keys, dtype, S, N, C, w, reps, reps, units_cap, it + 1 < n_iters, s,
                         track ? (it == 0 ? 1 : 2) : 0)))
      return st;
  }
  {
    const int64_t rows = S * C;
    finalize_kernel<<<(int)((rows + 3) / 4), 256, 0, s>>>(w.members, w.offsets, w.counts, perm, unit_start,
                                                          unit_size, units_cap, N, C, rows);
    LKV_CHECK_LAUNCH();
  }
  return LOUISKV_OK;
}

int check_common(const void* keys, int dtype, int64_t S, int N, int d, int C) {
  if (!keys) return fail(LOUISKV_ERR_NULL, "keys is NULL");
  if (dtype != LOUISKV_F32 && dtype != LOUISKV_BF16) return fail(LOUISKV_ERR_DTYPE, "unknown dtype %d", dtype);
  if (d != kHeadDim) return fail(LOUISKV_ERR_UNSUPPORTED, "head dim %d not supported (only 128)", d);
  if (S < 1 || N < 1) return fail(LOUISKV_ERR_SHAPE, "n_slices=%lld n_tokens=%d must be >= 1", (long long)S, N);
  if (C < 1 || C > N) return fail(LOUISKV_ERR_SHAPE, "n_clusters=%d must be in [1, n_tokens=%d]", C, N);
  if ((int64_t)S * ceil_div(N, kBf16KeysPerBlock) > (int64_t)INT32_MAX / 2 ||
      (int64_t)S * ceil_div(N, kF32KeysPerBlock) > (int64_t)INT32_MAX / 2)
    return fail(LOUISKV_ERR_SHAPE, "problem too large for one launch");
  return LOUISKV_OK;
}

}  // namespace
}  // namespace louiskv

using namespace louiskv;

extern "C" size_t louiskv_cluster_prefill_workspace_size(int64_t n_slices, int32_t n_tokens, int32_t d,
                                                         int32_t n_clusters, int32_t dtype) {
  (void)d;
  if (n_slices < 1 || n_tokens < 1 || n_clusters < 1) return 0;
  return carve(nullptr, n_slices, n_tokens, n_clusters, dtype == LOUISKV_BF16 ? LOUISKV_BF16 : LOUISKV_F32).bytes;
}

extern "C" int louiskv_cluster_prefill(const void* keys, int32_t dtype, int64_t n_slices, int32_t n_tokens,
                                       int32_t d, int32_t n_clusters, int32_t n_iters, const int32_t* init_idx,
                                       float* reps, int32_t units_cap, int32_t* unit_start, int32_t* unit_size,
                                       int32_t* assign, int32_t* perm, const void* values, void* k_pool,
                                       void* v_pool, int64_t pool_rows, int32_t pool_on_host,
                                       void* const* iter_events, void* workspace, size_t workspace_bytes,
                                       void* stream) {
  int st = check_common(keys, dtype, n_slices, n_tokens, d, n_clusters);
  if (st) return st;
  if (!init_idx || !reps || !unit_start || !unit_size || !assign || !perm)
    return fail(LOUISKV_ERR_NULL, "init_idx, reps, unit_start, unit_size, assign and perm are required");
  if (n_iters < 1) return fail(LOUISKV_ERR_SHAPE, "n_iters=%d must be >= 1", n_iters);
  if (units_cap < n_clusters) return fail(LOUISKV_ERR_SHAPE, "units_cap=%d < n_clusters=%d", units_cap, n_clusters);
  if (v_pool && !values) return fail(LOUISKV_ERR_NULL, "v_pool given without values");
  if ((k_pool || v_pool) && pool_rows < n_tokens)
    return fail(LOUISKV_ERR_SHAPE, "pool_rows=%lld < n_tokens=%d", (long long)pool_rows, n_tokens);
  if (pool_on_host && ((st = device_view_of_host_pool(k_pool, &k_pool)) || (st = device_view_of_host_pool(v_pool, &v_pool))))
    return st;
  const Ws need = carve(nullptr, n_slices, n_tokens, n_clusters, dtype);
  if (!workspace || workspace_bytes < need.bytes)
    return fail(LOUISKV_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need.bytes, workspace_bytes);
  const Ws w = carve(workspace, n_slices, n_tokens, n_clusters, dtype);
  hipStream_t s = as_stream(stream);
  if ((st = run_cluster(keys, dtype, n_slices, n_tokens, n_clusters, n_iters, init_idx, reps, units_cap, unit_start,
                        unit_size, assign, perm, iter_events, w, s)))
    return st;
  return launch_pack(keys, values, dtype, n_slices, n_tokens, perm, k_pool, v_pool, pool_rows, s);
}

namespace louiskv {
namespace {

size_t esize_of(int dtype) { return dtype == LOUISKV_BF16 ? 2 : 4; }

// Workspace of the pipelined prefill: the clustering workspace of one chunk,
// then (copy-engine writes only) one chunk of staged pool rows.
size_t pipelined_bytes(int64_t chunk, int N, int C, int dtype, bool staged) {
  size_t b = carve(nullptr, chunk, N, C, dtype).bytes;
  if (staged) b += align_up((size_t)chunk * N * kHeadDim * esize_of(dtype), 256);
  return b;
}

// Largest pack grid while the pack shares the chip with the clustering of
// the next chunk: enough rows in flight for the host link, few CUs held.
constexpr int kOverlapPackGrid = 256;

}  // namespace
}  // namespace louiskv

extern "C" size_t louiskv_cluster_prefill_pipelined_workspace_size(int64_t slices_per_chunk, int32_t n_tokens,
                                                                   int32_t d, int32_t n_clusters, int32_t dtype,
                                                                   int32_t pool_on_host, int32_t copy_engine) {
  (void)d;
  if (slices_per_chunk < 1 || n_tokens < 1 || n_clusters < 1) return 0;
  const int dt = dtype == LOUISKV_BF16 ? LOUISKV_BF16 : LOUISKV_F32;
  return pipelined_bytes(slices_per_chunk, n_tokens, n_clusters, dt, pool_on_host && copy_engine);
}

extern "C" int louiskv_cluster_prefill_pipelined(
    const void* keys, int32_t dtype, int64_t n_slices, int32_t n_tokens, int32_t d, int32_t n_clusters,
    int32_t n_iters, const int32_t* init_idx, float* reps, int32_t units_cap, int32_t* unit_start,
    int32_t* unit_size, int32_t* assign, int32_t* perm, const void* values, void* k_pool, void* v_pool,
    int64_t pool_rows, int32_t pool_on_host, int64_t slices_per_chunk, int32_t copy_engine,
    void* const* chunk_events, int64_t n_events, void* workspace, size_t workspace_bytes, void* stream,
    void* copy_stream) {
  int st = check_common(keys, dtype, n_slices, n_tokens, d, n_clusters);
  if (st) return st;
  if (!init_idx || !reps || !unit_start || !unit_size || !assign || !perm || !k_pool)
    return fail(LOUISKV_ERR_NULL, "init_idx, reps, unit_start, unit_size, assign, perm and k_pool are required");
  if (n_iters < 1) return fail(LOUISKV_ERR_SHAPE, "n_iters=%d must be >= 1", n_iters);
  if (units_cap < n_clusters) return fail(LOUISKV_ERR_SHAPE, "units_cap=%d < n_clusters=%d", units_cap, n_clusters);
  if (v_pool && !values) return fail(LOUISKV_ERR_NULL, "v_pool given without values");
  if (pool_rows < n_tokens)
    return fail(LOUISKV_ERR_SHAPE, "pool_rows=%lld < n_tokens=%d", (long long)pool_rows, n_tokens);
  if (slices_per_chunk < 1) return fail(LOUISKV_ERR_SHAPE, "slices_per_chunk=%lld must be >= 1",
                                        (long long)slices_per_chunk);
  const int64_t chunk = std::min(slices_per_chunk, n_slices);
  const int64_t n_chunks = (n_slices + chunk - 1) / chunk;
  if (!chunk_events || n_events < n_chunks + 1)
    return fail(LOUISKV_ERR_NULL, "chunk_events must hold n_chunks + 1 = %lld events, got %lld",
                (long long)(n_chunks + 1), (long long)n_events);
  for (int64_t i = 0; i <= n_chunks; ++i)
    if (!chunk_events[i]) return fail(LOUISKV_ERR_NULL, "chunk_events[%lld] is NULL", (long long)i);
  void* k_dev = k_pool;
  void* v_dev = v_pool;
  if (pool_on_host && ((st = device_view_of_host_pool(k_pool, &k_dev)) || (st = device_view_of_host_pool(v_pool, &v_dev))))
    return st;
  const bool staged = pool_on_host && copy_engine;
  const size_t need = pipelined_bytes(chunk, n_tokens, n_clusters, dtype, staged);
  if (!workspace || workspace_bytes < need)
    return fail(LOUISKV_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, workspace_bytes);
  const Ws w = carve(workspace, chunk, n_tokens, n_clusters, dtype);
  void* staging = static_cast<char*>(workspace) + w.bytes;
  hipStream_t s = as_stream(stream);
  hipStream_t cp = as_stream(copy_stream);
  const size_t es = esize_of(dtype);
  const size_t row_bytes = (size_t)kHeadDim * es;
  for (int64_t i = 0; i < n_chunks; ++i) {
    const int64_t c0 = i * chunk;
    const int64_t n = std::min(chunk, n_slices - c0);
    const size_t kv_off = (size_t)c0 * n_tokens * row_bytes;
    const size_t pool_off = (size_t)c0 * pool_rows * row_bytes;
    const void* keys_c = static_cast<const char*>(keys) + kv_off;
    const void* vals_c = values ? static_cast<const char*>(values) + kv_off : nullptr;
    int32_t* perm_c = perm + c0 * n_tokens;
    if ((st = run_cluster(keys_c, dtype, n, n_tokens, n_clusters, n_iters, init_idx + c0 * n_clusters,
                          reps + c0 * units_cap * kHeadDim, units_cap, unit_start + c0 * units_cap,
                          unit_size + c0 * units_cap, assign + c0 * n_tokens, perm_c, nullptr, w, s)))
      return st;
    // the pool write of this chunk waits for its clustering only and runs
    // beside the clustering of the next chunks
    LKV_CHECK_HIP(hipEventRecord(reinterpret_cast<hipEvent_t>(chunk_events[i]), s));
    LKV_CHECK_HIP(hipStreamWaitEvent(cp, reinterpret_cast<hipEvent_t>(chunk_events[i]), 0));
    if (!staged) {
      if ((st = launch_pack(keys_c, vals_c, dtype, n, n_tokens, perm_c,
                            static_cast<char*>(k_dev) + pool_off, v_dev ? static_cast<char*>(v_dev) + pool_off : nullptr,
                            pool_rows, cp, kOverlapPackGrid)))
        return st;
      continue;
    }
    // copy engine: permute into HBM staging, then one pitched copy over the host link
    for (int which = 0; which < 2; ++which) {
      void* host = which == 0 ? k_pool : v_pool;
      if (!host) continue;
      const void* src = which == 0 ? keys_c : vals_c;
      if ((st = launch_pack(src, nullptr, dtype, n, n_tokens, perm_c, staging, nullptr, n_tokens, cp))) return st;
      LKV_CHECK_HIP(hipMemcpy2DAsync(static_cast<char*>(host) + pool_off, (size_t)pool_rows * row_bytes, staging,
                                     (size_t)n_tokens * row_bytes, (size_t)n_tokens * row_bytes, (size_t)n,
                                     hipMemcpyDeviceToHost, cp));
    }
  }
  LKV_CHECK_HIP(hipEventRecord(reinterpret_cast<hipEvent_t>(chunk_events[n_chunks]), cp));
  LKV_CHECK_HIP(hipStreamWaitEvent(s, reinterpret_cast<hipEvent_t>(chunk_events[n_chunks]), 0));
  return LOUISKV_OK;
}

extern "C" int louiskv_page_prefill(const void* keys, const void* values, int32_t dtype, int64_t n_slices,
                                    int32_t n_tokens, int32_t d, int32_t page_len, float* reps, int32_t units_cap,
                                    int32_t* unit_start, int32_t* unit_size, void* k_pool, void* v_pool,
                                    int64_t pool_rows, int32_t pool_on_host, void* stream) {
  if (!keys || !reps || !unit_start || !unit_size)
    return fail(LOUISKV_ERR_NULL, "keys, reps, unit_start and unit_size are required");
  if (v_pool && !values) return fail(LOUISKV_ERR_NULL, "v_pool given without values");
  if (v_pool && !k_pool) return fail(LOUISKV_ERR_NULL, "v_pool given without k_pool");
  if (dtype != LOUISKV_F32 && dtype != LOUISKV_BF16) return fail(LOUISKV_ERR_DTYPE, "unknown dtype %d", dtype);
  if (d != kHeadDim) return fail(LOUISKV_ERR_UNSUPPORTED, "head dim %d not supported (only 128)", d);
  if (n_slices < 1 || n_tokens < 1 || page_len < 1)
    return fail(LOUISKV_ERR_SHAPE, "n_slices=%lld n_tokens=%d page_len=%d", (long long)n_slices, n_tokens, page_len);
  const int n_pages = ceil_div(n_tokens, page_len);
  if (units_cap < n_pages) return fail(LOUISKV_ERR_SHAPE, "units_cap=%d < %d pages", units_cap, n_pages);
  if (k_pool && pool_rows < n_tokens)
    return fail(LOUISKV_ERR_SHAPE, "pool_rows=%lld < n_tokens=%d", (long long)pool_rows, n_tokens);
  const int64_t items = n_slices * n_pages;
  if ((items + 3) / 4 > INT32_MAX) return fail(LOUISKV_ERR_SHAPE, "problem too large for one launch");
  int st;
  if (pool_on_host && ((st = device_view_of_host_pool(k_pool, &k_pool)) || (st = device_view_of_host_pool(v_pool, &v_pool))))
    return st;
  hipStream_t s = as_stream(stream);
  const unsigned grid = (unsigned)((items + 3) / 4);
  if (dtype == LOUISKV_BF16)
    page_units_kernel<uint16_t><<<grid, 256, 0, s>>>(static_cast<const uint16_t*>(keys),
                                                      static_cast<const uint16_t*>(values), n_tokens, page_len,
                                                      n_pages, items, reps, units_cap, unit_start, unit_size,
                                                      static_cast<uint16_t*>(k_pool), static_cast<uint16_t*>(v_pool),
                                                      pool_rows);
  else
    page_units_kernel<float><<<grid, 256, 0, s>>>(static_cast<const float*>(keys), static_cast<const float*>(values),
                                                   n_tokens, page_len, n_pages, items, reps, units_cap, unit_start,
                                                   unit_size, static_cast<float*>(k_pool), static_cast<float*>(v_pool),
                                                   pool_rows);
  LKV_CHECK_LAUNCH();
  return LOUISKV_OK;
}

extern "C" int louiskv_pack_pool(const void* keys, const void* values, int32_t dtype, int64_t n_slices,
                                 int32_t n_tokens, int32_t d, const int32_t* perm, void* k_pool, void* v_pool,
                                 int64_t pool_rows, int32_t pool_on_host, void* stream) {
  if (!keys || !perm || !k_pool) return fail(LOUISKV_ERR_NULL, "keys, perm and k_pool are required");
  if (v_pool && !values) return fail(LOUISKV_ERR_NULL, "v_pool given without values");
  if (dtype != LOUISKV_F32 && dtype != LOUISKV_BF16) return fail(LOUISKV_ERR_DTYPE, "unknown dtype %d", dtype);
  if (d != kHeadDim) return fail(LOUISKV_ERR_UNSUPPORTED, "head dim %d not supported (only 128)", d);
  if (n_slices < 1 || n_tokens < 1 || pool_rows < n_tokens)
    return fail(LOUISKV_ERR_SHAPE, "n_slices=%lld n_tokens=%d pool_rows=%lld", (long long)n_slices, n_tokens,
                (long long)pool_rows);
  int st;
  if (pool_on_host && ((st = device_view_of_host_pool(k_pool, &k_pool)) || (st = device_view_of_host_pool(v_pool, &v_pool))))
    return st;
  return launch_pack(keys, values, dtype, n_slices, n_tokens, perm, k_pool, v_pool, pool_rows, as_stream(stream));
}

extern "C" int louiskv_kmeans_assign(const void* keys, int32_t dtype, int64_t n_slices, int32_t n_tokens, int32_t d,
                                     int32_t n_clusters, const float* centroids, int32_t centroid_stride,
                                     int32_t* assign, void* workspace, size_t workspace_bytes, void* stream) {
  int st = check_common(keys, dtype, n_slices, n_tokens, d, n_clusters);
  if (st) return st;
  if (!centroids || !assign) return fail(LOUISKV_ERR_NULL, "centroids and assign are required");
  if (centroid_stride < n_clusters) return fail(LOUISKV_ERR_SHAPE, "centroid_stride < n_clusters");
  const Ws need = carve(nullptr, n_slices, n_tokens, n_clusters, dtype);
  if (!workspace || workspace_bytes < need.bytes)
    return fail(LOUISKV_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need.bytes, workspace_bytes);
  const Ws w = carve(workspace, n_slices, n_tokens, n_clusters, dtype);
  hipStream_t s = as_stream(stream);
  if ((st = launch_prep(centroids, centroid_stride, n_slices, n_clusters, dtype, w, false, s))) return st;
  return launch_assign(keys, dtype, n_slices, n_tokens, n_clusters, w, assign, false, false, 0, s);
}

extern "C" int louiskv_kmeans_update(const void* keys, int32_t dtype, int64_t n_slices, int32_t n_tokens, int32_t d,
                                     int32_t n_clusters, const int32_t* assign, const float* centroids_in,
                                     float* centroids_out, int32_t centroid_stride, int32_t* counts,
                                     void* workspace, size_t workspace_bytes, void* stream) {
  int st = check_common(keys, dtype, n_slices, n_tokens, d, n_clusters);
  if (st) return st;
  if (!assign || !centroids_in || !centroids_out) return fail(LOUISKV_ERR_NULL, "assign and centroids are required");
  if (centroid_stride < n_clusters) return fail(LOUISKV_ERR_SHAPE, "centroid_stride < n_clusters");
  const Ws need = carve(nullptr, n_slices, n_tokens, n_clusters, dtype);
  if (!workspace || workspace_bytes < need.bytes)
    return fail(LOUISKV_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need.bytes, workspace_bytes);
  const Ws w = carve(workspace, n_slices, n_tokens, n_clusters, dtype);
  hipStream_t s = as_stream(stream);
  {
    // a fill kernel rather than a memset node, so the call stays safe to capture
    const int64_t n = n_slices * n_clusters;
    fill_i32_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(w.counts, 0, n);
    LKV_CHECK_LAUNCH();
  }
  const int bps = ceil_div(n_tokens, kCountKeys);
  const bool lds_ok = (size_t)n_clusters * 4 <= kMaxHistLds;
  count_kernel<<<(unsigned)(n_slices * bps), 256, lds_ok ? (size_t)n_clusters * 4 : 0, s>>>(
      assign, w.counts, n_tokens, n_clusters, bps, lds_ok ? 1 : 0);
  LKV_CHECK_LAUNCH();
  if ((st = launch_scan_scatter(assign, n_slices, n_tokens, n_clusters, w, s))) return st;
  if ((st = launch_sum(keys, dtype, n_slices, n_tokens, n_clusters, w, centroids_in, centroids_out,
                       centroid_stride, false, s)))
    return st;
  if (counts)
    LKV_CHECK_HIP(hipMemcpyAsync(counts, w.counts, sizeof(int32_t) * n_slices * n_clusters,
                                 hipMemcpyDeviceToDevice, s));
  return LOUISKV_OK;
}
