/*
 * A plain C11 client of libboxconv (include/boxconv.h): no Python, no torch.
 *
 *   abi_client check   no GPU needed: ABI version, status strings, workspace
 *                      queries and argument validation (placeholder device
 *                      pointers that the library must reject before use).
 *   abi_client run     on a GPU: box_conv_fwd / box_conv_bwd through
 *                      hipMalloc'd buffers, checked against closed forms
 *                      computed here: the identity box returns the input
 *                      exactly (small integer-valued floats), a box covering
 *                      the whole map returns the map total at every pixel,
 *                      and the input gradient of that box is the total of the
 *                      upstream gradient at every pixel.
 * Prints "ok" and exits 0 on success; prints the failed check and exits 1.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "boxconv.h"

static int failures = 0;

#define EXPECT(cond)                                              \
  do {                                                            \
    if (!(cond)) {                                                \
      fprintf(stderr, "FAILED %s:%d: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                 \
    }                                                             \
  } while (0)

static int check(void) {
  void* fake = (void*)(uintptr_t)0x100000;      /* aligned, never dereferenced */
  void* fake_mis = (void*)(uintptr_t)0x100004;  /* misaligned */
  EXPECT(bc_abi_version() == 2);
  EXPECT(strcmp(bc_status_string(BC_OK), "ok") == 0);
  EXPECT(bc_status_string((bc_status)99) != NULL);
  /* pose-shaped layer: 32 x 256 maps of 64 x 48, 4 boxes; tables fit LDS, so
     the forward needs only the tap records (2 per box, 64 bytes each) */
  EXPECT(bc_box_workspace_bytes(0, 32, 256, 64, 48, 4, 0) == (size_t)2 * 256 * 4 * 64);
  EXPECT(bc_box_workspace_bytes(1, 32, 256, 64, 48, 4, 0) > (size_t)2 * 256 * 4 * 64);
  EXPECT(bc_box_workspace_bytes(0, 0, 256, 64, 48, 4, 0) == 0);
  EXPECT(bc_mix_workspace_bytes(BC_MIX_FWD, 32, 256, 1024, 3072, BC_BF16) == 0);
  EXPECT(bc_split_workspace_bytes(0, 32, 256, 64, 48, 4, BC_SPLIT_4) == (size_t)256 * 4 * 128);
  /* argument errors are returned before anything is launched */
  EXPECT(box_conv_fwd(NULL, BC_F32, fake, 1, 1, 8, 8, 1, fake, BC_F32, 0, NULL, 0, NULL) == BC_ERR_NULL);
  EXPECT(box_conv_fwd(fake, BC_F32, fake, 1, 0, 8, 8, 1, fake, BC_F32, 0, NULL, 0, NULL) == BC_ERR_SHAPE);
  EXPECT(box_conv_fwd(fake, BC_BF16, fake, 1, 1, 8, 8, 1, fake, BC_F32, 0, NULL, 0, NULL) == BC_ERR_DTYPE);
  EXPECT(box_conv_fwd(fake_mis, BC_F32, fake, 1, 1, 8, 8, 1, fake, BC_F32, 0, NULL, 0, NULL) == BC_ERR_ALIGN);
  EXPECT(box_conv_fwd(fake, BC_F32, fake, 1, 1, 8, 8, 1, fake, BC_F32, 0, NULL, 0, NULL) == BC_ERR_WORKSPACE);
  EXPECT(box_conv_fwd(fake, BC_F32, fake, 1, 1, 8, 8, 1, fake, BC_F32, 1u << 7, NULL, 0, NULL) == BC_ERR_UNSUPPORTED);
  EXPECT(box_conv_bwd(fake, fake, fake, 1, 1, 8, 8, 1, NULL, NULL, 0, NULL, 0, NULL) == BC_OK);
  EXPECT(box_conv_fwd_strided(fake, BC_F32, fake, 1, 1, 8, 8, 1, 0, fake, BC_F32, 0, NULL, 0, NULL) ==
         BC_ERR_SHAPE);
  EXPECT(sat_build(fake, BC_F32, fake, NULL, 1, 1, 8, 2000, NULL) == BC_ERR_SHAPE);
  EXPECT(box_conv_split_fwd(fake, fake, fake, 1, 1, 8, 8, 1, 9, fake, BC_F32, NULL, 0, NULL) ==
         BC_ERR_UNSUPPORTED);
  EXPECT(box_conv_split_fwd(fake, fake, fake, 1, 1, 8, 8, 1, BC_SPLIT_4 | BC_SPLIT_FORCE_HBM, fake, BC_F32, NULL, 0,
                            NULL) == BC_ERR_WORKSPACE);
  /* the masked bf16 input gradient: nothing requested is a no-op; rounded
     corners are refused (the mask needs x) */
  EXPECT(box_conv_bwd_relu_bf16(fake, fake, fake, 1, 1, 8, 8, 1, 1, NULL, NULL, 0, NULL, 0, NULL) == BC_OK);
  EXPECT(box_conv_bwd_relu_bf16(fake, fake, fake, 1, 1, 8, 8, 1, 1, fake, NULL, BC_FLAG_INTEGER_CORNERS, NULL, 0,
                                NULL) == BC_ERR_UNSUPPORTED);
  EXPECT(box_conv_bwd_relu_bf16(fake, fake, fake, 1, 1, 8, 8, 1, 1, fake, NULL, 0, NULL, 0, NULL) ==
         BC_ERR_WORKSPACE);
  EXPECT(bc_relu_grad_bf16(fake, fake, fake, 0, NULL) == BC_ERR_SHAPE);
  EXPECT(bc_relu_grad_bf16(fake, fake_mis, fake, 8, NULL) == BC_ERR_ALIGN);
  EXPECT(box_params_clip(NULL, 1, 1, NULL) == BC_ERR_NULL);
  EXPECT(pointwise_mix((bc_mix_mode)9, fake, BC_F32, fake, BC_F32, fake, BC_F32, 1, 8, 8, 8, BC_F32, 0, NULL, 0,
                       NULL, 0, NULL) == BC_ERR_UNSUPPORTED);
  /* sizes at and beyond the limits: the queries answer 0 and the calls
     refuse, with no arithmetic overflow on the way */
  EXPECT(bc_box_workspace_bytes(0, 1 << 16, 1 << 16, 1 << 16, 1 << 16, 1 << 16, 0) == 0);
  EXPECT(bc_box_workspace_bytes(1, 1, 1, 1 << 15, 1 << 15, 1, 0) > 0);
  EXPECT(bc_box_workspace_bytes(1, 2147483647, 1, 8, 8, 1, 0) == 0);
  EXPECT(bc_box_workspace_bytes(0, -1, 1, 8, 8, 1, 0) == 0);
  EXPECT(bc_box_workspace_bytes(2, 1, 1, 8, 8, 1, 0) == 0);
  EXPECT(bc_mix_workspace_bytes(BC_MIX_BWD_WEIGHT, 1 << 16, 1 << 16, 1 << 16, 1 << 16, BC_BF16) >= 0);
  EXPECT(box_conv_fwd(fake, BC_F32, fake, 2147483647, 2147483647, 8, 8, 1, fake, BC_F32, 0, fake, 1, NULL) ==
         BC_ERR_SHAPE);
  EXPECT(box_conv_bwd(fake, fake, fake, 1, 1, 1 << 16, 1 << 16, 1, fake, fake, 0, fake, 1, NULL) == BC_ERR_SHAPE);
  EXPECT(pointwise_mix(BC_MIX_FWD, fake, BC_F32, fake, BC_F32, fake, BC_F32, 1, 1 << 16, 1 << 16, 1 << 20, BC_F32,
                       0, NULL, 0, NULL, 0, NULL) == BC_ERR_SHAPE);
  EXPECT(pointwise_mix(BC_MIX_FWD, fake, BC_I32, fake, BC_F32, fake, BC_F32, 1, 8, 8, 8, BC_F32, 0, NULL, 0, NULL,
                       0, NULL) == BC_ERR_DTYPE);
  EXPECT(box_prep(fake, 1 << 15, 1 << 15, 0, fake, NULL) == BC_ERR_SHAPE);
  EXPECT(box_prep(fake, 4, 4, 1u << 9, fake, NULL) == BC_ERR_UNSUPPORTED);
  EXPECT(sat_build(fake, BC_BF16, fake, NULL, 1, 1, 8, 8, NULL) == BC_ERR_DTYPE);
  EXPECT(sat_build(fake, BC_I32, fake, fake, 1, 1, 8, 8, NULL) == BC_ERR_DTYPE);
  EXPECT(box_params_from_unit(fake, 4, 4, 0.f, 8.f, fake, NULL) == BC_ERR_SHAPE);
  EXPECT(box_params_unit_grad(fake, 4, 4, 8.f, 1e9f, fake, NULL) == BC_ERR_SHAPE);
  EXPECT(bc_cast_bf16(fake, fake_mis, 8, NULL) == BC_ERR_ALIGN);
  EXPECT(box_conv_split_bwd(fake, fake, fake, fake, 1, 1, 8, 8, 1, BC_SPLIT_2X, NULL, NULL, NULL, NULL, 0, NULL) ==
         BC_OK);
  EXPECT(box_conv_bwd_strided(fake, fake, fake, 1, 1, 8, 8, 1, 2000, fake, NULL, 0, NULL, 0, NULL) == BC_ERR_SHAPE);
  /* 256 x 256 maps: the streaming backward needs no table workspace, but a
     caller may still force the HBM tables */
  EXPECT(bc_box_workspace_bytes(1, 4, 128, 256, 256, 8, BC_FLAG_FORCE_HBM) >
         bc_box_workspace_bytes(1, 4, 128, 256, 256, 8, 0));
  /* the allocation-free backward refuses a workspace beyond its array before
     touching the device */
  EXPECT(bc_noalloc_scratch_bytes() == BC_NOALLOC_SCRATCH_BYTES);
  EXPECT(box_conv_bwd_noalloc(fake, fake, fake, 4, 128, 256, 256, 8, fake, fake, BC_FLAG_FORCE_HBM, NULL) ==
         BC_ERR_WORKSPACE);
  EXPECT(box_conv_bwd_noalloc(fake, fake, fake, 0, 1, 8, 8, 1, fake, fake, 0, NULL) == BC_ERR_SHAPE);
  return failures;
}

#define HIP_OK(call)                                                   \
  do {                                                                 \
    hipError_t e_ = (call);                                            \
    if (e_ != hipSuccess) {                                            \
      fprintf(stderr, "HIP error %d at %s:%d\n", (int)e_, __FILE__, __LINE__); \
      exit(1);                                                         \
    }                                                                  \
  } while (0)

static int run(void) {
  enum { N = 2, C = 3, H = 37, W = 29, B = 2 };
  const size_t nx = (size_t)N * C * H * W, ny = (size_t)N * C * B * H * W;
  float* hx = malloc(nx * sizeof(float));
  float* hg = malloc(ny * sizeof(float));
  float* hy = malloc(ny * sizeof(float));
  float* hgx = malloc(nx * sizeof(float));
  float hb[C * B * 4];
  for (size_t i = 0; i < nx; ++i) hx[i] = (float)((int)(i * 7919 % 17) - 8);
  for (size_t i = 0; i < ny; ++i) hg[i] = (float)((int)(i * 104729 % 13) - 6);
  for (int c = 0; c < C; ++c) {
    float* b0 = hb + (c * B + 0) * 4;  /* identity: the output pixel's own cell */
    float* b1 = hb + (c * B + 1) * 4;  /* covers every pixel of the map from everywhere */
    b0[0] = 0.f; b0[1] = 0.f; b0[2] = 0.5f; b0[3] = 0.5f;
    b1[0] = 0.f; b1[1] = 0.f; b1[2] = 1000.f; b1[3] = 1000.f;
  }
  float *dx, *db, *dy, *dg, *dgx;
  void *wsf, *wsb;
  const size_t nf = bc_box_workspace_bytes(0, N, C, H, W, B, 0);
  const size_t nb = bc_box_workspace_bytes(1, N, C, H, W, B, 0);
  HIP_OK(hipMalloc((void**)&dx, nx * sizeof(float)));
  HIP_OK(hipMalloc((void**)&dg, ny * sizeof(float)));
  HIP_OK(hipMalloc((void**)&dy, ny * sizeof(float)));
  HIP_OK(hipMalloc((void**)&dgx, nx * sizeof(float)));
  HIP_OK(hipMalloc((void**)&db, sizeof hb));
  HIP_OK(hipMalloc(&wsf, nf));
  HIP_OK(hipMalloc(&wsb, nb));
  HIP_OK(hipMemcpy(dx, hx, nx * sizeof(float), hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(dg, hg, ny * sizeof(float), hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(db, hb, sizeof hb, hipMemcpyHostToDevice));
  EXPECT(box_conv_fwd(dx, BC_F32, db, N, C, H, W, B, dy, BC_F32, 0, wsf, nf, NULL) == BC_OK);
  EXPECT(box_conv_bwd(dx, db, dg, N, C, H, W, B, dgx, NULL, 0, wsb, nb, NULL) == BC_OK);
  HIP_OK(hipDeviceSynchronize());
  HIP_OK(hipMemcpy(hy, dy, ny * sizeof(float), hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(hgx, dgx, nx * sizeof(float), hipMemcpyDeviceToHost));
  int bad_id = 0, bad_tot = 0, bad_gx = 0;
  for (int n = 0; n < N; ++n)
    for (int c = 0; c < C; ++c) {
      const float* xm = hx + ((size_t)n * C + c) * H * W;
      const float* y0 = hy + (((size_t)n * C + c) * B + 0) * H * W;
      const float* y1 = hy + (((size_t)n * C + c) * B + 1) * H * W;
      double tot = 0.0;
      for (int i = 0; i < H * W; ++i) tot += xm[i];
      for (int i = 0; i < H * W; ++i) {
        if (y0[i] != xm[i]) ++bad_id;
        if (fabs(y1[i] - tot) > 1e-4 * (1.0 + fabs(tot))) ++bad_tot;
      }
      /* input gradient: identity box passes g0 through; the covering box
         spreads the total of g1 over every pixel */
      const float* g0 = hg + (((size_t)n * C + c) * B + 0) * H * W;
      const float* g1 = hg + (((size_t)n * C + c) * B + 1) * H * W;
      double gt = 0.0;
      for (int i = 0; i < H * W; ++i) gt += g1[i];
      const float* gx = hgx + ((size_t)n * C + c) * H * W;
      for (int i = 0; i < H * W; ++i)
        if (fabs(gx[i] - (g0[i] + gt)) > 1e-4 * (1.0 + fabs(gt))) ++bad_gx;
    }
  EXPECT(bad_id == 0);
  EXPECT(bad_tot == 0);
  EXPECT(bad_gx == 0);
  hipFree(dx); hipFree(dg); hipFree(dy); hipFree(dgx); hipFree(db); hipFree(wsf); hipFree(wsb);
  free(hx); free(hg); free(hy); free(hgx);
  return failures;
}

int main(int argc, char** argv) {
  const char* mode = argc > 1 ? argv[1] : "check";
  const int f = strcmp(mode, "run") == 0 ? run() : check();
  if (f) return 1;
  printf("ok\n");
  return 0;
}
