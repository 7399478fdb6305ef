/*
 * mafat_c_caller.c -- a plain C program that drives libmafat through its C
 * ABI only (include/mafat.h and the HIP runtime; no Python, no torch): the
 * boundary test of the GPU suite (tests/test_gpu_c_caller.py).
 *
 * Usage: mafat_c_caller DIR
 *   DIR/config.txt   "in_h in_w in_c batch dtype n_layers n_groups flags", then
 *                    one line "op c_out f s p act" per layer, then one line
 *                    "group_start rows cols" per group (flags: the plan flags
 *                    of mafat_plan_create_flags, 0 for mafat_plan_create)
 *   DIR/x.bin        the input, NHWC, batch frames, in the run dtype
 *   DIR/w<l>.bin     conv layer l's weights [c_out][f][f][c_in] in the dtype
 *   DIR/s<l>.bin     its float32 scale, DIR/b<l>.bin its float32 bias
 * Writes DIR/y.bin (the network output, in the dtype) and DIR/regions.txt
 * (every group's tile regions as mafat_plan_regions reports them).
 *
 * Steps: plan, workspace size, caller-owned device buffers (hipMalloc), the
 * weights of every layer that the plan packs repacked by mafat_pack_weights
 * into buffers of mafat_packed_weights_size bytes, mafat_run_network on a
 * stream of its own, then the same network group by
 * group through mafat_run_group into a second output, which must equal the
 * first bit for bit; a workspace one byte too small must be refused with
 * MAFAT_EWORKSPACE and a message, before any launch.  Exit status 0 on
 * success, 1 on any failure (with a message on stderr).
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "mafat.h"

#define MAXL 64
#define MAXG 16

static int fail(const char* what, int rc) {
  fprintf(stderr, "mafat_c_caller: %s failed: %d (%s) %s\n", what, rc, mafat_status_string(rc), mafat_last_error());
  return 1;
}

static int hip_ok(hipError_t e, const char* what) {
  if (e != hipSuccess) {
    fprintf(stderr, "mafat_c_caller: %s: %s\n", what, hipGetErrorString(e));
    return 0;
  }
  return 1;
}

/* Reads a whole file of exactly `bytes` bytes into a new host buffer. */
static void* read_file(const char* dir, const char* name, size_t bytes) {
  char path[1024];
  snprintf(path, sizeof(path), "%s/%s", dir, name);
  FILE* f = fopen(path, "rb");
  if (!f) { fprintf(stderr, "mafat_c_caller: cannot open %s\n", path); return NULL; }
  void* p = malloc(bytes ? bytes : 1);
  size_t got = p ? fread(p, 1, bytes, f) : 0;
  int extra = fgetc(f);
  fclose(f);
  if (!p || got != bytes || extra != EOF) {
    fprintf(stderr, "mafat_c_caller: %s: expected %zu bytes\n", path, bytes);
    free(p);
    return NULL;
  }
  return p;
}

/* Copies a host file to a new device buffer. */
static void* upload(const char* dir, const char* name, size_t bytes) {
  void* h = read_file(dir, name, bytes);
  if (!h) return NULL;
  void* d = NULL;
  if (!hip_ok(hipMalloc(&d, bytes), "hipMalloc") || !hip_ok(hipMemcpy(d, h, bytes, hipMemcpyHostToDevice), "copy in")) {
    free(h);
    return NULL;
  }
  free(h);
  return d;
}

int main(int argc, char** argv) {
  if (argc != 2) { fprintf(stderr, "usage: mafat_c_caller DIR\n"); return 1; }
  const char* dir = argv[1];
  char path[1024];
  snprintf(path, sizeof(path), "%s/config.txt", dir);
  FILE* cf = fopen(path, "r");
  if (!cf) { fprintf(stderr, "mafat_c_caller: cannot open %s\n", path); return 1; }
  int in_h, in_w, in_c, batch, dtype, nl, ng, flags;
  mafat_layer layers[MAXL];
  int32_t gs[MAXG], rows[MAXG], cols[MAXG];
  int ok = fscanf(cf, "%d %d %d %d %d %d %d %d", &in_h, &in_w, &in_c, &batch, &dtype, &nl, &ng, &flags) == 8 &&
           nl >= 1 && nl <= MAXL && ng >= 1 && ng <= MAXG;
  for (int l = 0; ok && l < nl; ++l) {
    mafat_layer* L = &layers[l];
    ok = fscanf(cf, "%d %d %d %d %d %d", &L->op, &L->c_out, &L->f, &L->s, &L->p, &L->act) == 6;
  }
  for (int g = 0; ok && g < ng; ++g) ok = fscanf(cf, "%d %d %d", &gs[g], &rows[g], &cols[g]) == 3;
  fclose(cf);
  if (!ok) { fprintf(stderr, "mafat_c_caller: bad config.txt\n"); return 1; }
  const size_t esz = dtype == MAFAT_BF16 ? 2 : 4;

  mafat_plan* plan = NULL;
  int rc = flags ? mafat_plan_create_flags(layers, nl, in_h, in_w, in_c, gs, ng, rows, cols, flags, &plan)
                 : mafat_plan_create(layers, nl, in_h, in_w, in_c, gs, ng, rows, cols, &plan);
  if (rc != MAFAT_OK) return fail("mafat_plan_create", rc);

  /* shapes: the input of every layer, the output of the last and of every group */
  int32_t dims[MAXL][6];
  for (int l = 0; l < nl; ++l)
    if ((rc = mafat_plan_layer_shape(plan, l, dims[l])) != MAFAT_OK) return fail("mafat_plan_layer_shape", rc);

  /* regions of every group, as text */
  snprintf(path, sizeof(path), "%s/regions.txt", dir);
  FILE* rf = fopen(path, "w");
  if (!rf) { fprintf(stderr, "mafat_c_caller: cannot write %s\n", path); return 1; }
  for (int g = 0; g < ng; ++g) {
    int32_t nt = 0;
    if ((rc = mafat_plan_num_tiles(plan, g, &nt)) != MAFAT_OK) return fail("mafat_plan_num_tiles", rc);
    const int gl = ((g + 1 < ng) ? gs[g + 1] : nl) - gs[g];
    const int64_t cap = (int64_t)nt * gl;
    mafat_rect* ir = (mafat_rect*)malloc(sizeof(mafat_rect) * (size_t)cap);
    mafat_rect* orr = (mafat_rect*)malloc(sizeof(mafat_rect) * (size_t)cap);
    if (!ir || !orr) return 1;
    if ((rc = mafat_plan_regions(plan, g, ir, orr, cap)) != MAFAT_OK) return fail("mafat_plan_regions", rc);
    for (int64_t k = 0; k < cap; ++k)
      fprintf(rf, "%d %lld %d %d %d %d %d %d %d %d\n", g, (long long)k, ir[k].y0, ir[k].y1, ir[k].x0, ir[k].x1,
              orr[k].y0, orr[k].y1, orr[k].x0, orr[k].x1);
    free(ir);
    free(orr);
  }
  fclose(rf);

  /* caller-owned device buffers */
  const size_t x_bytes = (size_t)batch * in_h * in_w * in_c * esz;
  const size_t y_elems = (size_t)batch * dims[nl - 1][3] * dims[nl - 1][4] * dims[nl - 1][5];
  void* x = upload(dir, "x.bin", x_bytes);
  if (!x) return 1;
  void* w[MAXL];
  float* sc[MAXL];
  float* bi[MAXL];
  for (int l = 0; l < nl; ++l) {
    w[l] = NULL; sc[l] = NULL; bi[l] = NULL;
    if (layers[l].op != MAFAT_CONV) continue;
    const size_t wn = (size_t)dims[l][5] * layers[l].f * layers[l].f * dims[l][2];
    char name[64];
    snprintf(name, sizeof(name), "w%d.bin", l);
    if (!(w[l] = upload(dir, name, wn * esz))) return 1;
    snprintf(name, sizeof(name), "s%d.bin", l);
    if (!(sc[l] = (float*)upload(dir, name, (size_t)dims[l][5] * 4))) return 1;
    snprintf(name, sizeof(name), "b%d.bin", l);
    if (!(bi[l] = (float*)upload(dir, name, (size_t)dims[l][5] * 4))) return 1;
  }
  void* cuts[MAXG];
  void* cuts2[MAXG];
  for (int g = 0; g + 1 < ng; ++g) {
    const int last = gs[g + 1] - 1;
    const size_t n = (size_t)batch * dims[last][3] * dims[last][4] * dims[last][5] * esz;
    if (!hip_ok(hipMalloc(&cuts[g], n), "hipMalloc cut") || !hip_ok(hipMalloc(&cuts2[g], n), "hipMalloc cut"))
      return 1;
  }
  void *y = NULL, *y2 = NULL, *ws = NULL;
  size_t ws_bytes = 0;
  if ((rc = mafat_workspace_size(plan, batch, dtype, &ws_bytes)) != MAFAT_OK) return fail("mafat_workspace_size", rc);
  if (!hip_ok(hipMalloc(&y, y_elems * esz), "hipMalloc y") || !hip_ok(hipMalloc(&y2, y_elems * esz), "hipMalloc y") ||
      !hip_ok(hipMalloc(&ws, ws_bytes ? ws_bytes : 256), "hipMalloc workspace"))
    return 1;
  hipStream_t stream;
  if (!hip_ok(hipStreamCreate(&stream), "hipStreamCreate")) return 1;

  /* layers whose weights the plan takes packed: repack them on the stream */
  void* wk[MAXL];
  for (int l = 0; l < nl; ++l) {
    wk[l] = NULL;
    if (layers[l].op != MAFAT_CONV) continue;
    size_t pb = 0;
    if ((rc = mafat_packed_weights_size(plan, l, dtype, &pb)) != MAFAT_OK) return fail("mafat_packed_weights_size", rc);
    if (pb == 0) continue;
    void* packed = NULL;
    if (!hip_ok(hipMalloc(&packed, pb), "hipMalloc packed weights")) return 1;
    if ((rc = mafat_pack_weights(plan, l, dtype, w[l], packed, stream)) != MAFAT_OK)
      return fail("mafat_pack_weights", rc);
    wk[l] = w[l];
    w[l] = packed;
  }

  /* a workspace one byte short is refused before anything is enqueued */
  if (ws_bytes > 0) {
    rc = mafat_run_network(plan, batch, dtype, x, y, cuts, (const void* const*)w, (const float* const*)sc,
                           (const float* const*)bi, ws, ws_bytes - 1, stream);
    if (rc != MAFAT_EWORKSPACE || strlen(mafat_last_error()) == 0) {
      fprintf(stderr, "mafat_c_caller: a short workspace gave %d, not MAFAT_EWORKSPACE\n", rc);
      return 1;
    }
  }

  /* the whole network */
  rc = mafat_run_network(plan, batch, dtype, x, y, cuts, (const void* const*)w, (const float* const*)sc,
                         (const float* const*)bi, ws, ws_bytes, stream);
  if (rc != MAFAT_OK) return fail("mafat_run_network", rc);
  /* the same, group by group: group g reads the previous group's output */
  for (int g = 0; g < ng; ++g) {
    const void* gin = (g == 0) ? x : cuts2[g - 1];
    void* gout = (g + 1 < ng) ? cuts2[g] : y2;
    rc = mafat_run_group(plan, g, batch, dtype, gin, gout, (const void* const*)w, (const float* const*)sc,
                         (const float* const*)bi, ws, ws_bytes, stream);
    if (rc != MAFAT_OK) return fail("mafat_run_group", rc);
  }
  if (!hip_ok(hipStreamSynchronize(stream), "stream synchronisation")) return 1;

  unsigned char* hy = (unsigned char*)malloc(y_elems * esz);
  unsigned char* hy2 = (unsigned char*)malloc(y_elems * esz);
  if (!hy || !hy2) return 1;
  if (!hip_ok(hipMemcpy(hy, y, y_elems * esz, hipMemcpyDeviceToHost), "copy out") ||
      !hip_ok(hipMemcpy(hy2, y2, y_elems * esz, hipMemcpyDeviceToHost), "copy out"))
    return 1;
  if (memcmp(hy, hy2, y_elems * esz) != 0) {
    fprintf(stderr, "mafat_c_caller: mafat_run_group per group differs from mafat_run_network\n");
    return 1;
  }
  snprintf(path, sizeof(path), "%s/y.bin", dir);
  FILE* yf = fopen(path, "wb");
  if (!yf || fwrite(hy, 1, y_elems * esz, yf) != y_elems * esz) { fprintf(stderr, "cannot write y.bin\n"); return 1; }
  fclose(yf);

  free(hy);
  free(hy2);
  hipStreamDestroy(stream);
  for (int l = 0; l < nl; ++l) { hipFree(w[l]); hipFree(wk[l]); hipFree(sc[l]); hipFree(bi[l]); }
  for (int g = 0; g + 1 < ng; ++g) { hipFree(cuts[g]); hipFree(cuts2[g]); }
  hipFree(x); hipFree(y); hipFree(y2); hipFree(ws);
  mafat_plan_destroy(plan);
  printf("mafat_c_caller: ok (%d layers, %d groups, batch %d, %s, flags %d)\n", nl, ng, batch,
         dtype == MAFAT_BF16 ? "bf16" : "f32", flags);
  return 0;
}
