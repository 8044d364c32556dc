/*
 * A plain C caller of the library: the k-means prefill and a decode loop
 * (boundary test, retrieval as a pool row list, window store, attention)
 * through include/louiskv.h alone, with device memory from the HIP runtime's
 * C API.  Test infrastructure: tests/test_gpu_c_abi.py writes the inputs,
 * runs this program and compares what it writes with the same calls made
 * through the Python binding.
 *
 *   abi_example DIR     reads DIR/meta.txt and DIR/*.bin, writes DIR/out_*.bin
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "louiskv.h"

#define CHECK_HIP(x)                                                              \
  do {                                                                            \
    hipError_t e_ = (x);                                                          \
    if (e_ != hipSuccess) {                                                       \
      fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));             \
      exit(2);                                                                    \
    }                                                                             \
  } while (0)

#define CHECK_LKV(x)                                                              \
  do {                                                                            \
    int s_ = (x);                                                                 \
    if (s_ != LOUISKV_OK) {                                                       \
      fprintf(stderr, "%s failed: %s (%s)\n", #x, louiskv_status_str(s_),        \
              louiskv_last_error());                                              \
      exit(3);                                                                    \
    }                                                                             \
  } while (0)

static void* read_file(const char* dir, const char* name, size_t bytes) {
  char path[4096];
  snprintf(path, sizeof path, "%s/%s", dir, name);
  FILE* f = fopen(path, "rb");
  if (!f) { fprintf(stderr, "cannot open %s\n", path); exit(4); }
  void* p = malloc(bytes);
  if (fread(p, 1, bytes, f) != bytes) { fprintf(stderr, "short read %s\n", path); exit(4); }
  fclose(f);
  return p;
}

static void write_file(const char* dir, const char* name, const void* p, size_t bytes) {
  char path[4096];
  snprintf(path, sizeof path, "%s/%s", dir, name);
  FILE* f = fopen(path, "wb");
  if (!f || fwrite(p, 1, bytes, f) != bytes) { fprintf(stderr, "cannot write %s\n", path); exit(4); }
  fclose(f);
}

static void* to_device(const void* host, size_t bytes) {
  void* d = NULL;
  CHECK_HIP(hipMalloc(&d, bytes ? bytes : 1));
  if (host && bytes) CHECK_HIP(hipMemcpy(d, host, bytes, hipMemcpyHostToDevice));
  return d;
}

static void* zeros(size_t bytes) {
  void* d = to_device(NULL, bytes);
  CHECK_HIP(hipMemset(d, 0, bytes ? bytes : 1));
  return d;
}

int main(int argc, char** argv) {
  if (argc != 2) { fprintf(stderr, "usage: %s DIR\n", argv[0]); return 1; }
  const char* dir = argv[1];
  char mpath[4096];
  snprintf(mpath, sizeof mpath, "%s/meta.txt", dir);
  FILE* mf = fopen(mpath, "r");
  if (!mf) { fprintf(stderr, "cannot open %s\n", mpath); return 4; }
  int S, N, C, iters, T, W, seg, B, G, HQ, HKV;
  double tau;
  if (fscanf(mf, "%d %d %d %d %d %d %d %d %d %d %d %lf", &S, &N, &C, &iters, &T, &W, &seg, &B, &G, &HQ, &HKV,
             &tau) != 12) { fprintf(stderr, "bad meta\n"); return 4; }
  fclose(mf);
  const int D = 128, g = HQ / HKV;
  const int cap = C + (T > W ? (T - W + seg - 1) / seg : 0);
  const int pool_rows = N + T;
  const size_t row = (size_t)D * 2;   /* bf16 */

  uint16_t* hk = read_file(dir, "keys.bin", (size_t)S * N * row);
  uint16_t* hv = read_file(dir, "values.bin", (size_t)S * N * row);
  int32_t* hinit = read_file(dir, "init.bin", (size_t)S * C * 4);
  uint16_t* hq = read_file(dir, "queries.bin", (size_t)T * G * HQ * row);
  uint16_t* hgk = read_file(dir, "gen_keys.bin", (size_t)T * S * row);
  uint16_t* hgv = read_file(dir, "gen_values.bin", (size_t)T * S * row);

  void* keys = to_device(hk, (size_t)S * N * row);
  void* values = to_device(hv, (size_t)S * N * row);
  int32_t* init = to_device(hinit, (size_t)S * C * 4);
  float* reps = zeros((size_t)S * cap * D * 4);
  int32_t* ustart = zeros((size_t)S * cap * 4);
  int32_t* usize = zeros((size_t)S * cap * 4);
  int32_t* assign = zeros((size_t)S * N * 4);
  int32_t* perm = zeros((size_t)S * N * 4);
  void* kpool = zeros((size_t)S * pool_rows * row);
  void* vpool = zeros((size_t)S * pool_rows * row);
  size_t wsb = louiskv_cluster_prefill_workspace_size(S, N, D, C, LOUISKV_BF16);
  void* ws = zeros(wsb);
  CHECK_LKV(louiskv_cluster_prefill(keys, LOUISKV_BF16, S, N, D, C, iters, init, reps, cap, ustart, usize, assign,
                                    perm, values, kpool, vpool, pool_rows, 0, NULL, ws, wsb, NULL));

  void* q = to_device(NULL, (size_t)G * HQ * row);
  void* knew = to_device(NULL, (size_t)S * row);
  void* vnew = to_device(NULL, (size_t)S * row);
  void* qref = zeros((size_t)G * HQ * row);
  uint8_t* fire = zeros(G);
  double* r = zeros((size_t)G * 8);
  void* kloc = zeros((size_t)S * W * row);
  void* vloc = zeros((size_t)S * W * row);
  int32_t* sel_units = zeros((size_t)S * cap * 4);
  int32_t* n_sel_units = zeros((size_t)S * 4);
  int32_t* n_sel = zeros((size_t)S * 4);
  int32_t* sel_rows = zeros((size_t)S * B * 4);
  size_t rwsb = louiskv_retrieve_rows_workspace_size(S, cap);
  void* rws = zeros(rwsb);
  size_t awsb = louiskv_sparse_decode_attn_rows_workspace_size(S, g, D, B, W);
  void* aws = zeros(awsb);
  float* out = zeros((size_t)G * HQ * D * 4);
  float* lse = zeros((size_t)G * HQ * 4);
  float* hout = malloc((size_t)T * G * HQ * D * 4);

  for (int t = 0; t < T; ++t) {
    CHECK_HIP(hipMemcpy(q, hq + (size_t)t * G * HQ * D, (size_t)G * HQ * row, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(knew, hgk + (size_t)t * S * D, (size_t)S * row, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(vnew, hgv + (size_t)t * S * D, (size_t)S * row, hipMemcpyHostToDevice));
    int32_t ev, n_ev, n_local, local_start, n_ev_before = 0;
    if (t > 0) CHECK_LKV(louiskv_window_info(t - 1, W, seg, &ev, &n_ev_before, NULL, NULL));
    CHECK_LKV(louiskv_boundary_check(q, qref, LOUISKV_BF16, G, HQ, D, tau, LOUISKV_REF_ANCHOR, t == 0, r, fire,
                                     NULL));
    CHECK_LKV(louiskv_retrieve_rows(q, LOUISKV_BF16, S, HKV, g, D, 1.0 / 11.313708498984761, reps, ustart, usize,
                                    cap, C + n_ev_before, B, fire, sel_units, n_sel_units, n_sel, sel_rows, NULL,
                                    rws, rwsb, NULL));
    CHECK_LKV(louiskv_segment_output(knew, vnew, LOUISKV_BF16, S, D, kloc, vloc, W, t, seg, reps, ustart, usize,
                                     cap, C, kpool, vpool, pool_rows, N, 0, NULL));
    CHECK_LKV(louiskv_window_info(t, W, seg, &ev, &n_ev, &n_local, &local_start));
    CHECK_LKV(louiskv_sparse_decode_attn_rows(q, LOUISKV_BF16, S, HKV, g, D, (float)(1.0 / 11.313708498984761),
                                              kpool, vpool, pool_rows, sel_rows, n_sel, B, kloc, vloc, W,
                                              local_start, n_local, out, LOUISKV_F32, lse, aws, awsb, NULL));
    CHECK_HIP(hipMemcpy(hout + (size_t)t * G * HQ * D, out, (size_t)G * HQ * D * 4, hipMemcpyDeviceToHost));
  }
  CHECK_HIP(hipDeviceSynchronize());

  /* the same decode through louiskv_decode_step (boundary, store, retrieval
     and attention of a step in one call), from a fresh prefill */
  float* reps2 = zeros((size_t)S * cap * D * 4);
  int32_t* ustart2 = zeros((size_t)S * cap * 4);
  int32_t* usize2 = zeros((size_t)S * cap * 4);
  int32_t* assign2 = zeros((size_t)S * N * 4);
  int32_t* perm2 = zeros((size_t)S * N * 4);
  void* kpool2 = zeros((size_t)S * pool_rows * row);
  void* vpool2 = zeros((size_t)S * pool_rows * row);
  void* ws2 = zeros(wsb);
  CHECK_LKV(louiskv_cluster_prefill(keys, LOUISKV_BF16, S, N, D, C, iters, init, reps2, cap, ustart2, usize2,
                                    assign2, perm2, values, kpool2, vpool2, pool_rows, 0, NULL, ws2, wsb, NULL));
  void* qref2 = zeros((size_t)G * HQ * row);
  uint8_t* fire2 = zeros(G);
  double* r2 = zeros((size_t)G * 8);
  void* kloc2 = zeros((size_t)S * W * row);
  void* vloc2 = zeros((size_t)S * W * row);
  int32_t* sel_units2 = zeros((size_t)S * cap * 4);
  int32_t* n_sel_units2 = zeros((size_t)S * 4);
  int32_t* n_sel2 = zeros((size_t)S * 4);
  int32_t* sel_rows2 = zeros((size_t)S * B * 4);
  size_t swsb = louiskv_decode_step_workspace_size(S, LOUISKV_BF16, g, cap, B, W);
  if (swsb == 0) {
    fprintf(stderr, "louiskv_decode_step_workspace_size returned 0\n");
    return 1;
  }
  void* sws = zeros(swsb);   /* zero before the first call; every call leaves its counters at zero */
  float* out2 = zeros((size_t)G * HQ * D * 4);
  float* lse2 = zeros((size_t)G * HQ * 4);
  float* hout2 = malloc((size_t)T * G * HQ * D * 4);
  for (int t = 0; t < T; ++t) {
    CHECK_HIP(hipMemcpy(q, hq + (size_t)t * G * HQ * D, (size_t)G * HQ * row, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(knew, hgk + (size_t)t * S * D, (size_t)S * row, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(vnew, hgv + (size_t)t * S * D, (size_t)S * row, hipMemcpyHostToDevice));
    CHECK_LKV(louiskv_decode_step(q, qref2, LOUISKV_BF16, G, HQ, HKV, D, tau, LOUISKV_REF_ANCHOR, t, r2, fire2,
                                  knew, vnew, kloc2, vloc2, W, seg, reps2, ustart2, usize2, cap, C, kpool2, vpool2,
                                  pool_rows, N, B, sel_units2, n_sel_units2, n_sel2, sel_rows2, NULL, out2,
                                  LOUISKV_F32, lse2, sws, swsb, NULL));
    CHECK_HIP(hipMemcpy(hout2 + (size_t)t * G * HQ * D, out2, (size_t)G * HQ * D * 4, hipMemcpyDeviceToHost));
  }
  CHECK_HIP(hipDeviceSynchronize());
  write_file(dir, "out_attn_step.bin", hout2, (size_t)T * G * HQ * D * 4);

  int32_t* hassign = malloc((size_t)S * N * 4);
  float* hreps = malloc((size_t)S * cap * D * 4);
  CHECK_HIP(hipMemcpy(hassign, assign, (size_t)S * N * 4, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(hreps, reps, (size_t)S * cap * D * 4, hipMemcpyDeviceToHost));
  write_file(dir, "out_assign.bin", hassign, (size_t)S * N * 4);
  write_file(dir, "out_reps.bin", hreps, (size_t)S * cap * D * 4);
  write_file(dir, "out_attn.bin", hout, (size_t)T * G * HQ * D * 4);
  printf("abi_example: %d slices, %d tokens, %d clusters, %d decode steps done (per-stage calls and "
         "louiskv_decode_step)\n", S, N, C, T);
  return 0;
}
