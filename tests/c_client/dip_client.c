/* dip_client.c -- a plain C caller of the library's C ABI (no Python, no
 * torch): reads an instance and a batch of candidate orders from a file,
 * copies the orders to device memory with the HIP runtime, runs
 * dip_sim_create / dip_sim_evaluate / dip_sim_argmin, and writes the four
 * outputs and the argmin key to a second file.
 *
 * Input file (little endian):
 *   int32 P, N, E, n_slots; int64 stride, n_cand;
 *   int32 n_ops[P]; int32 pred_ptr[N+1]; int32 pred_op[E]; uint8 op_kind[N];
 *   int32 op_slot[N]; int32 mem_cap[P]; int32 op_cost[N]; int32 edge_comm[E];
 *   int32 slot_act[n_slots]; int16 orders[n_cand][stride].
 * Output file: int32 makespan[n]; int32 bubble[n][P]; int32 peak[n][P];
 *   uint8 flags[n]; uint64 argmin key.
 * Exit status 0 on success; otherwise the failing call and its message go to
 * stderr. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <hip/hip_runtime_api.h>

#include "dip_sim.h"

static int fail(const char *what, const char *msg) {
  fprintf(stderr, "dip_client: %s: %s\n", what, msg);
  return 1;
}

static void *read_n(FILE *f, size_t elem, size_t n) {
  void *p = malloc(elem * (n ? n : 1));
  if (p && n && fread(p, elem, n, f) != n) {
    free(p);
    return NULL;
  }
  return p;
}

#define HIP_CHECK(call)                                              \
  do {                                                               \
    hipError_t e_ = (call);                                          \
    if (e_ != hipSuccess) return fail(#call, hipGetErrorString(e_)); \
  } while (0)

#define DIP_CHECK(call)                                   \
  do {                                                    \
    int rc_ = (call);                                     \
    if (rc_ != DIP_OK) return fail(#call, dip_sim_strerror(rc_)); \
  } while (0)

int main(int argc, char **argv) {
  if (argc != 3) return fail("usage", "dip_client IN OUT");
  if (dip_sim_abi_version() != DIP_SIM_ABI_VERSION) return fail("abi", "version mismatch");
  FILE *in = fopen(argv[1], "rb");
  if (!in) return fail("fopen", argv[1]);
  int32_t hdr[4];
  int64_t hdr64[2];
  if (fread(hdr, 4, 4, in) != 4 || fread(hdr64, 8, 2, in) != 2) return fail("read", "header");
  const int32_t P = hdr[0], N = hdr[1], E = hdr[2], n_slots = hdr[3];
  const int64_t stride = hdr64[0], n = hdr64[1];
  if (P < 1 || N < 0 || E < 0 || n_slots < 0 || stride < 8 || n < 0) return fail("read", "sizes");
  int32_t *n_ops = read_n(in, 4, (size_t)P);
  int32_t *pred_ptr = read_n(in, 4, (size_t)N + 1);
  int32_t *pred_op = read_n(in, 4, (size_t)E);
  uint8_t *op_kind = read_n(in, 1, (size_t)N);
  int32_t *op_slot = read_n(in, 4, (size_t)N);
  int32_t *mem_cap = read_n(in, 4, (size_t)P);
  int32_t *op_cost = read_n(in, 4, (size_t)N);
  int32_t *edge_comm = read_n(in, 4, (size_t)E);
  int32_t *slot_act = read_n(in, 4, (size_t)n_slots);
  int16_t *orders = read_n(in, 2, (size_t)(n * stride));
  fclose(in);
  if (!n_ops || !pred_ptr || !pred_op || !op_kind || !op_slot || !mem_cap || !op_cost ||
      !edge_comm || !slot_act || !orders)
    return fail("read", "arrays");

  dip_topology topo = {P, n_ops, pred_ptr, pred_op, op_kind, op_slot, n_slots, mem_cap, stride};
  dip_costs costs = {op_cost, edge_comm, slot_act};
  DIP_CHECK(dip_sim_check_topology(&topo));
  DIP_CHECK(dip_sim_check_costs(&topo, &costs));
  dip_sim *h = NULL;
  DIP_CHECK(dip_sim_create(&topo, &h));

  /* device buffers: orders in, four outputs and the key out */
  const size_t nz = (size_t)(n ? n : 1);
  int16_t *d_orders = NULL;
  int32_t *d_ms = NULL, *d_bub = NULL, *d_pk = NULL;
  uint8_t *d_fl = NULL;
  uint64_t *d_key = NULL;
  HIP_CHECK(hipMalloc((void **)&d_orders, 2 * nz * (size_t)stride));
  HIP_CHECK(hipMalloc((void **)&d_ms, 4 * nz));
  HIP_CHECK(hipMalloc((void **)&d_bub, 4 * nz * (size_t)P));
  HIP_CHECK(hipMalloc((void **)&d_pk, 4 * nz * (size_t)P));
  HIP_CHECK(hipMalloc((void **)&d_fl, nz));
  HIP_CHECK(hipMalloc((void **)&d_key, 8));
  HIP_CHECK(hipMemcpy(d_orders, orders, 2 * (size_t)(n * stride), hipMemcpyHostToDevice));
  const uint64_t none = ~(uint64_t)0;
  HIP_CHECK(hipMemcpy(d_key, &none, 8, hipMemcpyHostToDevice));

  hipStream_t s;
  HIP_CHECK(hipStreamCreate(&s));
  DIP_CHECK(dip_sim_evaluate(h, &costs, d_orders, n, d_ms, d_bub, d_pk, d_fl, (void *)s));
  DIP_CHECK(dip_sim_argmin(h, d_ms, d_fl, n, 0, d_key, (void *)s));
  HIP_CHECK(hipStreamSynchronize(s));

  int32_t *ms = malloc(4 * nz), *bub = malloc(4 * nz * (size_t)P), *pk = malloc(4 * nz * (size_t)P);
  uint8_t *fl = malloc(nz);
  uint64_t key = 0;
  if (!ms || !bub || !pk || !fl) return fail("malloc", "outputs");
  HIP_CHECK(hipMemcpy(ms, d_ms, 4 * (size_t)n, hipMemcpyDeviceToHost));
  HIP_CHECK(hipMemcpy(bub, d_bub, 4 * (size_t)(n * P), hipMemcpyDeviceToHost));
  HIP_CHECK(hipMemcpy(pk, d_pk, 4 * (size_t)(n * P), hipMemcpyDeviceToHost));
  HIP_CHECK(hipMemcpy(fl, d_fl, (size_t)n, hipMemcpyDeviceToHost));
  HIP_CHECK(hipMemcpy(&key, d_key, 8, hipMemcpyDeviceToHost));

  FILE *out = fopen(argv[2], "wb");
  if (!out) return fail("fopen", argv[2]);
  if (fwrite(ms, 4, (size_t)n, out) != (size_t)n ||
      fwrite(bub, 4, (size_t)(n * P), out) != (size_t)(n * P) ||
      fwrite(pk, 4, (size_t)(n * P), out) != (size_t)(n * P) ||
      fwrite(fl, 1, (size_t)n, out) != (size_t)n || fwrite(&key, 8, 1, out) != 1)
    return fail("write", argv[2]);
  fclose(out);

  dip_sim_destroy(h);
  HIP_CHECK(hipStreamDestroy(s));
  hipFree(d_orders);
  hipFree(d_ms);
  hipFree(d_bub);
  hipFree(d_pk);
  hipFree(d_fl);
  hipFree(d_key);
  printf("dip_client: %lld candidates, key %llu\n", (long long)n, (unsigned long long)key);
  return 0;
}
