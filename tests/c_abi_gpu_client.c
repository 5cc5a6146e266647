/* A plain C99 program that runs the GPU path through libemu.so with the HIP runtime's C API only (no
 * Python, no torch): the tiny decoder's TP1 PP1 -> TP2 PP1 reshard, then pack into 12,288-byte buckets
 * and unpack into a receiver set. Source element e of tensor i holds a fixed hash of (i, e) that the
 * test regenerates. Writes the destination tensors (dst.bin) and the buckets (buckets.bin), each
 * concatenated in table order, into the directory given as the first argument, and prints
 * "key value" lines. */
#include <hip/hip_runtime_api.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "emu.h"

#define HIPCHECK(call)                                                        \
  do {                                                                        \
    hipError_t e_ = (call);                                                   \
    if (e_ != hipSuccess) {                                                   \
      fprintf(stderr, "%s -> %s\n", #call, hipGetErrorString(e_));            \
      return 1;                                                               \
    }                                                                         \
  } while (0)
#define EMUCHECK(call)                                                                      \
  do {                                                                                      \
    int rc_ = (call);                                                                       \
    if (rc_ != EMU_OK) {                                                                    \
      fprintf(stderr, "%s -> %s: %s\n", #call, emu_status_str(rc_), emu_last_error());      \
      return 1;                                                                             \
    }                                                                                       \
  } while (0)

static emu_layout_t tiny(int tp) {
  emu_layout_t l;
  l.model.num_layers = 2; l.model.hidden = 256; l.model.num_heads = 4; l.model.num_kv_heads = 2;
  l.model.head_dim = 64; l.model.ffn_hidden = 688; l.model.vocab = 1024;
  l.tp = tp; l.pp = 1; l.vocab_pad_multiple = 0;
  l.dtype = EMU_BF16; l.qkv_format = EMU_QKV_HEAD_INTERLEAVED; l.mlp_format = EMU_GATE_UP_BLOCK;
  return l;
}

static int write_all(const char* dir, const char* name, void** bufs, const uint64_t* sizes, int n) {
  char path[4096];
  FILE* f;
  int i;
  snprintf(path, sizeof path, "%s/%s", dir, name);
  f = fopen(path, "wb");
  if (!f) return 1;
  for (i = 0; i < n; ++i) {
    void* h = malloc(sizes[i] ? sizes[i] : 1);
    if (!h || hipMemcpy(h, bufs[i], sizes[i], hipMemcpyDeviceToHost) != hipSuccess ||
        fwrite(h, 1, sizes[i], f) != sizes[i]) {
      fclose(f);
      return 1;
    }
    free(h);
  }
  return fclose(f) != 0;
}

int main(int argc, char** argv) {
  emu_layout_t a = tiny(1), b = tiny(2);
  emu_plan_t plan = NULL;
  emu_plan_info_t info;
  emu_tensor_desc_t d;
  const uint64_t B = 12288;
  uint64_t nb = 0, sb = 0, k;
  int32_t i, ns, nd;
  emu_bucket_desc_t* bk;
  void **S, **D, **R, **K, *ws, *ws2;
  uint64_t *ssz, *dsz, *ksz, *hs, *hd, *hr, *hk, *d_sp, *d_dp, *d_rp, *d_kp;
  int equal = 1;

  if (argc < 2) return 2;
  EMUCHECK(emu_plan(&a, &b, &plan));
  EMUCHECK(emu_plan_info(plan, &info));
  ns = info.n_src_tensors;
  nd = info.n_dst_tensors;
  S = calloc((size_t)ns, sizeof(void*)); D = calloc((size_t)nd, sizeof(void*)); R = calloc((size_t)nd, sizeof(void*));
  ssz = calloc((size_t)ns, 8); dsz = calloc((size_t)nd, 8);
  hs = calloc((size_t)ns, 8); hd = calloc((size_t)nd, 8); hr = calloc((size_t)nd, 8);
  if (!S || !D || !R || !ssz || !dsz || !hs || !hd || !hr) return 1;
  for (i = 0; i < ns; ++i) {
    uint16_t* h;
    uint64_t e;
    EMUCHECK(emu_tensor_info(plan, 0, i, &d));
    ssz[i] = d.bytes;
    h = malloc(d.bytes);
    if (!h) return 1;
    for (e = 0; e < d.bytes / 2; ++e)
      h[e] = (uint16_t)((((uint32_t)i * 2654435761u) ^ ((uint32_t)e * 40503u)) & 0xffffu);
    HIPCHECK(hipMalloc(&S[i], d.bytes));
    HIPCHECK(hipMemcpy(S[i], h, d.bytes, hipMemcpyHostToDevice));
    free(h);
    hs[i] = (uint64_t)(uintptr_t)S[i];
  }
  for (i = 0; i < nd; ++i) {
    EMUCHECK(emu_tensor_info(plan, 1, i, &d));
    dsz[i] = d.bytes;
    HIPCHECK(hipMalloc(&D[i], d.bytes));
    HIPCHECK(hipMalloc(&R[i], d.bytes));
    HIPCHECK(hipMemset(D[i], 0xA5, d.bytes));
    HIPCHECK(hipMemset(R[i], 0x5A, d.bytes));
    hd[i] = (uint64_t)(uintptr_t)D[i];
    hr[i] = (uint64_t)(uintptr_t)R[i];
  }
  EMUCHECK(emu_check_tables(plan, hs, hd));
  HIPCHECK(hipMalloc((void**)&d_sp, (size_t)ns * 8));
  HIPCHECK(hipMalloc((void**)&d_dp, (size_t)nd * 8));
  HIPCHECK(hipMalloc((void**)&d_rp, (size_t)nd * 8));
  HIPCHECK(hipMemcpy(d_sp, hs, (size_t)ns * 8, hipMemcpyHostToDevice));
  HIPCHECK(hipMemcpy(d_dp, hd, (size_t)nd * 8, hipMemcpyHostToDevice));
  HIPCHECK(hipMemcpy(d_rp, hr, (size_t)nd * 8, hipMemcpyHostToDevice));

  HIPCHECK(hipMalloc(&ws, info.workspace_bytes));
  HIPCHECK(hipMalloc(&ws2, info.workspace_bytes));
  printf("not_uploaded %s\n", emu_status_str(emu_reshard(plan, ws2, d_sp, d_dp, NULL)));
  HIPCHECK(hipMemset(ws, 0, info.workspace_bytes));
  EMUCHECK(emu_plan_upload(plan, ws, info.workspace_bytes, NULL));
  {
    /* the uploaded workspace, tables built on the device included, against the host's image of it */
    uint8_t* want = malloc((size_t)info.workspace_bytes);
    uint8_t* got = malloc((size_t)info.workspace_bytes);
    if (!want || !got) return 1;
    EMUCHECK(emu_plan_workspace_image(plan, want, info.workspace_bytes));
    HIPCHECK(hipMemcpy(got, ws, info.workspace_bytes, hipMemcpyDeviceToHost));
    printf("upload_image_equal %d\n", memcmp(want, got, (size_t)info.workspace_bytes) == 0);
    free(want);
    free(got);
  }
  EMUCHECK(emu_reshard(plan, ws, d_sp, d_dp, NULL));

  /* buckets of every destination rank, rank 0 first, sized as the library reports them */
  EMUCHECK(emu_bucket_layout(plan, 1, B, -1, &nb, &sb));
  K = calloc((size_t)nb, sizeof(void*)); ksz = calloc((size_t)nb, 8); hk = calloc((size_t)nb, 8);
  bk = calloc((size_t)nb, sizeof(emu_bucket_desc_t));
  if (!K || !ksz || !hk || !bk) return 1;
  EMUCHECK(emu_bucket_info(plan, 1, B, 0, nb, bk));
  for (k = 0; k < nb; ++k) {
    ksz[k] = bk[k].bytes;
    HIPCHECK(hipMalloc(&K[k], ksz[k]));
    hk[k] = (uint64_t)(uintptr_t)K[k];
  }
  EMUCHECK(emu_check_bucket_tables(plan, 1, B, hd, hk));
  HIPCHECK(hipMalloc((void**)&d_kp, (size_t)nb * 8));
  HIPCHECK(hipMemcpy(d_kp, hk, (size_t)nb * 8, hipMemcpyHostToDevice));
  EMUCHECK(emu_pack_buckets(plan, ws, 1, B, d_dp, d_kp, NULL));
  EMUCHECK(emu_unpack_buckets(plan, ws, 1, B, d_kp, d_rp, NULL));
  HIPCHECK(hipDeviceSynchronize());

  for (i = 0; i < nd && equal; ++i) {
    void* x = malloc(dsz[i]);
    void* y = malloc(dsz[i]);
    if (!x || !y) return 1;
    HIPCHECK(hipMemcpy(x, D[i], dsz[i], hipMemcpyDeviceToHost));
    HIPCHECK(hipMemcpy(y, R[i], dsz[i], hipMemcpyDeviceToHost));
    equal = memcmp(x, y, dsz[i]) == 0;
    free(x);
    free(y);
  }
  if (write_all(argv[1], "dst.bin", D, dsz, nd) || write_all(argv[1], "buckets.bin", K, ksz, (int)nb)) return 1;
  printf("tensors %d %d\n", ns, nd);
  printf("buckets %llu\n", (unsigned long long)nb);
  printf("unpack_equal %d\n", equal);
  {
    /* the receiver's own plan over the same buckets: destination layout to itself, read from buckets */
    emu_plan_t rp = NULL;
    emu_plan_info_t ri;
    void* wsr;
    int requal = 1;
    EMUCHECK(emu_plan_from_buckets(&b, &b, B, &rp));
    EMUCHECK(emu_plan_info(rp, &ri));
    if ((uint64_t)ri.n_src_tensors != nb || ri.n_dst_tensors != nd) return 1;
    HIPCHECK(hipMalloc(&wsr, ri.workspace_bytes));
    EMUCHECK(emu_plan_upload(rp, wsr, ri.workspace_bytes, NULL));
    for (i = 0; i < nd; ++i) HIPCHECK(hipMemset(R[i], 0x11, dsz[i]));
    EMUCHECK(emu_reshard(rp, wsr, d_kp, d_rp, NULL));
    HIPCHECK(hipDeviceSynchronize());
    for (i = 0; i < nd && requal; ++i) {
      void* x = malloc(dsz[i]);
      void* y = malloc(dsz[i]);
      if (!x || !y) return 1;
      HIPCHECK(hipMemcpy(x, D[i], dsz[i], hipMemcpyDeviceToHost));
      HIPCHECK(hipMemcpy(y, R[i], dsz[i], hipMemcpyDeviceToHost));
      requal = memcmp(x, y, dsz[i]) == 0;
      free(x);
      free(y);
    }
    printf("receiver_equal %d\n", requal);
    HIPCHECK(hipFree(wsr));
    EMUCHECK(emu_plan_free(rp));
  }

  for (i = 0; i < ns; ++i) HIPCHECK(hipFree(S[i]));
  for (i = 0; i < nd; ++i) {
    HIPCHECK(hipFree(D[i]));
    HIPCHECK(hipFree(R[i]));
  }
  for (k = 0; k < nb; ++k) HIPCHECK(hipFree(K[k]));
  free(bk);
  HIPCHECK(hipFree(d_sp)); HIPCHECK(hipFree(d_dp)); HIPCHECK(hipFree(d_rp)); HIPCHECK(hipFree(d_kp));
  HIPCHECK(hipFree(ws)); HIPCHECK(hipFree(ws2));
  EMUCHECK(emu_plan_free(plan));
  free(S); free(D); free(R); free(K); free(ssz); free(dsz); free(ksz); free(hs); free(hd); free(hr); free(hk);
  printf("done 1\n");
  return 0;
}
