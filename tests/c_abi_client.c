/* A plain C99 client of libemu.so: compiled by tests/test_c_abi.py with gcc -std=c99 -Wall -Werror
 * against include/emu.h, it uses the host-only half of the ABI (no GPU): layout checks, the 8B copy
 * map and its tensor inventory, the host-side pointer-table check, and the transition-DAG planner on
 * the section 6.1 example. It prints one "key value" line per fact for the test to compare. */
#include <stdio.h>
#include <stdlib.h>

#include "emu.h"

#define CHECK(call)                                                                         \
  do {                                                                                      \
    int rc_ = (call);                                                                       \
    if (rc_ != EMU_OK) {                                                                    \
      fprintf(stderr, "%s -> %s: %s\n", #call, emu_status_str(rc_), emu_last_error());      \
      return 1;                                                                             \
    }                                                                                       \
  } while (0)

static emu_layout_t layout(int tp, int pp) {
  emu_layout_t l;
  l.model.num_layers = 32; l.model.hidden = 4096; l.model.num_heads = 32; l.model.num_kv_heads = 8;
  l.model.head_dim = 128; l.model.ffn_hidden = 14336; l.model.vocab = 128256;
  l.tp = tp; l.pp = pp; l.vocab_pad_multiple = 0;
  l.dtype = EMU_BF16; l.qkv_format = EMU_QKV_HEAD_INTERLEAVED; l.mlp_format = EMU_GATE_UP_BLOCK;
  return l;
}

int main(void) {
  emu_layout_t src = layout(2, 2), dst = layout(4, 1), bad = layout(3, 1);
  emu_plan_t plan = NULL;
  emu_plan_info_t info;
  emu_tensor_desc_t d;
  uint64_t *sp, *dp, a;
  int32_t i;

  printf("version %d\n", emu_version());
  printf("bad_layout %s\n", emu_status_str(emu_layout_check(&bad)));
  CHECK(emu_plan(&src, &dst, &plan));
  CHECK(emu_plan_info(plan, &info));
  printf("tensors %d %d\n", info.n_src_tensors, info.n_dst_tensors);
  printf("bytes %llu %llu\n", (unsigned long long)info.bytes_read, (unsigned long long)info.bytes_written);
  CHECK(emu_tensor_info(plan, 1, 1, &d));
  printf("dst1 %d %d %lld %lld\n", d.rank, d.kind, (long long)d.rows, (long long)d.cols);

  /* host copies of pointer tables: every tensor in its own 256-byte aligned slot */
  sp = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)info.n_src_tensors);
  dp = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)info.n_dst_tensors);
  if (!sp || !dp) return 1;
  a = 1ull << 32;
  for (i = 0; i < info.n_src_tensors; ++i) {
    CHECK(emu_tensor_info(plan, 0, i, &d));
    sp[i] = a;
    a = (a + d.bytes + 255) / 256 * 256;
  }
  for (i = 0; i < info.n_dst_tensors; ++i) {
    CHECK(emu_tensor_info(plan, 1, i, &d));
    dp[i] = a;
    a = (a + d.bytes + 255) / 256 * 256;
  }
  CHECK(emu_check_tables(plan, sp, dp));
  dp[7] = sp[3];
  printf("overlap %s\n", emu_status_str(emu_check_tables(plan, sp, dp)));
  free(sp);
  free(dp);
  {
    /* buckets of the destination side at B = 2^28, sized by the library */
    uint64_t nb = 0, sb = 0, k, sum = 0;
    emu_bucket_desc_t* bk;
    CHECK(emu_bucket_layout(plan, 1, 1ull << 28, -1, &nb, &sb));
    bk = (emu_bucket_desc_t*)malloc(sizeof(emu_bucket_desc_t) * (size_t)nb);
    if (!bk) return 1;
    CHECK(emu_bucket_info(plan, 1, 1ull << 28, 0, nb, bk));
    for (k = 0; k < nb; ++k) sum += bk[k].bytes;
    printf("buckets %llu %llu %d %llu %llu\n", (unsigned long long)nb, (unsigned long long)sum, bk[nb - 1].rank,
           (unsigned long long)bk[nb - 1].index, (unsigned long long)bk[nb - 1].bytes);
    printf("bucket_range %s\n", emu_status_str(emu_bucket_info(plan, 1, 1ull << 28, nb, 1, bk)));
    free(bk);
  }
  {
    /* the receiver's plan: its source side is the source ranks' 2^28-byte buckets */
    emu_plan_t rp = NULL;
    emu_plan_info_t ri;
    uint64_t nb = 0, sb = 0;
    CHECK(emu_plan_from_buckets(&src, &dst, 1ull << 28, &rp));
    CHECK(emu_plan_info(rp, &ri));
    CHECK(emu_bucket_layout(plan, 0, 1ull << 28, -1, &nb, &sb));
    printf("receiver %d %d %llu %d\n", ri.n_src_tensors, ri.n_dst_tensors, (unsigned long long)nb,
           ri.bytes_written == info.bytes_written);
    CHECK(emu_plan_free(rp));
    printf("receiver_odd %s\n", emu_status_str(emu_plan_from_buckets(&src, &dst, 3, &rp)));
  }
  {
    /* the workspace image: refused for a buffer one byte short, filled for a whole one */
    uint8_t* img = (uint8_t*)malloc((size_t)info.workspace_bytes);
    uint64_t k, nz = 0;
    if (!img) return 1;
    printf("image_short %s\n", emu_status_str(emu_plan_workspace_image(plan, img, info.workspace_bytes - 1)));
    CHECK(emu_plan_workspace_image(plan, img, info.workspace_bytes));
    for (k = 0; k < info.workspace_bytes; ++k) nz += img[k] != 0;
    printf("image_nonzero %d\n", nz > 0);
    free(img);
  }
  CHECK(emu_plan_free(plan));
  printf("freed_again %s\n", emu_status_str(emu_plan_free(plan)));

  {
    /* a PP-only change with resident shards aliased: nothing left to copy */
    emu_layout_t s2 = layout(4, 2), d2 = layout(4, 1);
    CHECK(emu_plan_ex(&s2, &d2, EMU_PLAN_ALIAS_RESIDENT, &plan));
    CHECK(emu_plan_info(plan, &info));
    printf("alias %d %d %llu %llu %lld\n", info.n_alias_tensors, info.aliased, (unsigned long long)info.alias_bytes,
           (unsigned long long)info.bytes_read, (long long)info.n_tiles);
    CHECK(emu_plan_free(plan));
  }

  /* transition DAG: one training model-stage, (TP4, PP8) on 32 GPUs -> (TP8, PP2) on the first 16 */
  {
    int32_t gpus[32], tgt[16];
    emu_stage_transition_t st;
    emu_link_model_t links;
    emu_dag_t dag = NULL;
    emu_dag_info_t di;
    for (i = 0; i < 32; ++i) gpus[i] = i;
    for (i = 0; i < 16; ++i) tgt[i] = i;
    st.kind = EMU_STAGE_TRAINING; st.tp = 4; st.pp = 8; st.dp = 1;
    st.tgt_tp = 8; st.tgt_pp = 2; st.tgt_dp = 1; st.reserved = 0;
    st.gpus = gpus; st.tgt_gpus = tgt; st.state_bytes = 3200.0;
    links.gpus_per_node = 8; links.reserved = 0;
    links.intra_bw = 100.0; links.inter_bw = 10.0; links.hbm_bw = 1000.0; links.setup_s = 0.5;
    CHECK(emu_dag_plan(&st, 1, &links, &dag));
    CHECK(emu_dag_info(dag, &di));
    printf("dag %d %d %.6f\n", di.n_nodes, di.n_edges, di.l_tran_s);
    CHECK(emu_dag_free(dag));
  }
  return 0;
}
