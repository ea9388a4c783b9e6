/*
 * Plain C client of the LayerCheck C interface: no Python, no torch.  It
 * allocates the model arrays with hipMalloc, runs the decision step of every
 * step of a recorded trajectory (score, select, pack into a fresh device
 * version buffer), then loses the live state and rebuilds it with the
 * composite restore, writing everything the library returned to a file that
 * the test compares with the oracle.  Every version is also appended to a
 * persistence store with the overlapped append (a reuse event, the stream
 * never waits), and the composite rebuilt from the store must equal the one
 * rebuilt from the device versions byte for byte.  At every step the
 * allocation-free score (lc_score_layers_static) of the same arrays must
 * equal the context's u bit for bit.
 *
 *   lc_c_client <input file> <output file> <store directory>
 *
 * Input (little endian):
 *   "LCC1", u32 n_layers, u32 n_segments, u32 weight_dtype, u32 has_master,
 *   u32 mode, u32 n_steps, i64 s_max, i64 t_base, i64 t_fail, f64 eps_w,
 *   f64 k0[n_layers], f64 lr_scale[n_steps + 1],
 *   per segment: u32 layer, u32 zero, u64 numel,
 *   then n_steps + 1 states (step t_base, t_base + 1, ...), each the weights
 *   (all segments back to back, weight dtype), then the master (if present),
 *   m and v (fp32).
 * Output:
 *   per layer: u64 numel, u64 record bytes;
 *   base version: u64 bytes, payload;
 *   per step: f64 u[N], f64 delta[N], i64 t_last[N], u8 mask[N],
 *             u32 n_selected, u32 n_forced, u64 payload_bytes, i64 max_age,
 *             f64 weighted_age, u64 bytes, payload;
 *   after the restore: i64 chosen[N], i64 t_last[N], then W, S, master (if
 *   present), m, v.
 * Exit status 0 on success; on failure the message goes to stderr.
 */
#include <hip/hip_runtime_api.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "layercheck.h"

static FILE *out_f;

static void die(const char *what) {
  fprintf(stderr, "lc_c_client: %s\n", what);
  exit(1);
}

#define LC(call)                                                                \
  do {                                                                          \
    lc_status st_ = (call);                                                     \
    if (st_ != LC_OK) {                                                         \
      fprintf(stderr, "lc_c_client: %s -> %d: %s\n", #call, (int)st_, lc_last_error()); \
      exit(1);                                                                  \
    }                                                                           \
  } while (0)

#define HIP(call)                                                                      \
  do {                                                                                 \
    hipError_t e_ = (call);                                                            \
    if (e_ != hipSuccess) {                                                            \
      fprintf(stderr, "lc_c_client: %s -> %s\n", #call, hipGetErrorString(e_));        \
      exit(1);                                                                         \
    }                                                                                  \
  } while (0)

static void rd(FILE *f, void *p, size_t n) {
  if (n && fread(p, 1, n, f) != n) die("short input file");
}

static void wr(const void *p, size_t n) {
  if (n && fwrite(p, 1, n, out_f) != n) die("short write");
}

static void *xmalloc(size_t n) {
  void *p = malloc(n ? n : 1);
  if (!p) die("out of host memory");
  return p;
}

/* A device copy of the payload of one pack, kept as a version. */
typedef struct {
  int64_t step;
  uint8_t *mask;
  void *payload;
  uint64_t bytes;
} version_t;

/* Packs the pending selection into a new device buffer of exactly its size
 * (one call: the capacity is the whole payload) and writes it out. */
static version_t pack_version(lc_ctx *c, int64_t step, const uint8_t *mask, uint32_t N, const uint64_t *rec) {
  version_t v;
  uint64_t need = 0;
  for (uint32_t l = 0; l < N; ++l)
    if (mask[l]) need += rec[l];
  v.step = step;
  v.mask = (uint8_t *)xmalloc(N);
  memcpy(v.mask, mask, N);
  v.bytes = need;
  v.payload = NULL;
  if (need) HIP(hipMalloc(&v.payload, need));
  lc_pack_result r;
  LC(lc_pack_selected(c, v.payload, need, 0, &r));
  if (r.bytes_written != need || !r.done) die("one pack call should hold the whole selection");
  HIP(hipDeviceSynchronize());
  uint8_t *h = (uint8_t *)xmalloc(need);
  if (need) HIP(hipMemcpy(h, v.payload, need, hipMemcpyDeviceToHost));
  wr(&need, 8);
  wr(h, need);
  free(h);
  return v;
}

/* Copies the live arrays to fresh host buffers. */
static uint8_t *snapshot(const uint8_t *d, size_t n) {
  uint8_t *h = (uint8_t *)xmalloc(n);
  HIP(hipMemcpy(h, d, n, hipMemcpyDeviceToHost));
  return h;
}

int main(int argc, char **argv) {
  if (argc != 4) die("usage: lc_c_client <input> <output> <store directory>");
  FILE *in = fopen(argv[1], "rb");
  if (!in) die("cannot open the input");
  out_f = fopen(argv[2], "wb");
  if (!out_f) die("cannot open the output");

  char magic[4];
  rd(in, magic, 4);
  if (memcmp(magic, "LCC1", 4)) die("bad magic");
  uint32_t N, S, dtype, has_master, mode, n_steps;
  int64_t s_max, t_base, t_fail;
  double eps_w;
  rd(in, &N, 4);
  rd(in, &S, 4);
  rd(in, &dtype, 4);
  rd(in, &has_master, 4);
  rd(in, &mode, 4);
  rd(in, &n_steps, 4);
  rd(in, &s_max, 8);
  rd(in, &t_base, 8);
  rd(in, &t_fail, 8);
  rd(in, &eps_w, 8);
  double *k0 = (double *)xmalloc(8 * N);
  double *lr_scale = (double *)xmalloc(8 * (n_steps + 1));
  rd(in, k0, 8 * N);
  rd(in, lr_scale, 8 * (n_steps + 1));
  const size_t esz = dtype == LC_DT_BF16 ? 2 : 4;

  lc_segment *segs = (lc_segment *)xmalloc(sizeof(lc_segment) * S);
  uint64_t total = 0;
  for (uint32_t i = 0; i < S; ++i) {
    memset(&segs[i], 0, sizeof(segs[i]));
    uint32_t zero;
    rd(in, &segs[i].layer, 4);
    rd(in, &zero, 4);
    rd(in, &segs[i].numel, 8);
    total += segs[i].numel;
  }
  /* one device allocation per array, segments back to back (each 256-B aligned
   * offset would also do; packing them tightly exercises unaligned segments) */
  uint8_t *dW, *dS, *dM = NULL, *dm, *dv;
  HIP(hipMalloc((void **)&dW, total * esz));
  HIP(hipMalloc((void **)&dS, total * esz));
  if (has_master) HIP(hipMalloc((void **)&dM, total * 4));
  HIP(hipMalloc((void **)&dm, total * 4));
  HIP(hipMalloc((void **)&dv, total * 4));
  uint64_t off = 0;
  for (uint32_t i = 0; i < S; ++i) {
    segs[i].weight = dW + off * esz;
    segs[i].shadow = dS + off * esz;
    segs[i].master = has_master ? (float *)(dM + off * 4) : NULL;
    segs[i].exp_avg = (float *)(dm + off * 4);
    segs[i].exp_avg_sq = (float *)(dv + off * 4);
    off += segs[i].numel;
  }
  uint8_t *hW = (uint8_t *)xmalloc(total * esz), *hM = (uint8_t *)xmalloc(total * 4);
  uint8_t *hm = (uint8_t *)xmalloc(total * 4), *hv = (uint8_t *)xmalloc(total * 4);

  /* loads the next recorded state into the device arrays */
#define LOAD_STATE()                                                     \
  do {                                                                   \
    rd(in, hW, total * esz);                                             \
    if (has_master) rd(in, hM, total * 4);                               \
    rd(in, hm, total * 4);                                               \
    rd(in, hv, total * 4);                                               \
    HIP(hipMemcpy(dW, hW, total * esz, hipMemcpyHostToDevice));          \
    if (has_master) HIP(hipMemcpy(dM, hM, total * 4, hipMemcpyHostToDevice)); \
    HIP(hipMemcpy(dm, hm, total * 4, hipMemcpyHostToDevice));            \
    HIP(hipMemcpy(dv, hv, total * 4, hipMemcpyHostToDevice));            \
  } while (0)

  hipStream_t stream;
  HIP(hipStreamCreate(&stream));
  lc_layout_desc d;
  memset(&d, 0, sizeof(d));
  d.n_layers = N;
  d.n_segments = S;
  d.segments = segs;
  d.weight_dtype = (int32_t)dtype;
  d.has_master = (int32_t)has_master;
  d.mode = (int32_t)mode;
  d.k0 = k0;
  d.s_max = s_max;
  d.eps_w = eps_w;
  d.t_base = t_base;
  d.stream = stream;

  uint64_t *numel = (uint64_t *)xmalloc(8 * N), *rec = (uint64_t *)xmalloc(8 * N);
  LC(lc_query_layout(&d, numel, rec));
  for (uint32_t l = 0; l < N; ++l) {
    wr(&numel[l], 8);
    wr(&rec[l], 8);
  }
  LOAD_STATE();
  lc_ctx *c = NULL;
  LC(lc_init_layout(&d, &c));
  for (uint32_t l = 0; l < N; ++l)
    if (lc_record_bytes(c, l) != rec[l]) die("lc_record_bytes disagrees with lc_query_layout");

  lc_store *store = NULL;
  LC(lc_store_open(argv[3], N, rec, 8u << 20, &store));
  hipEvent_t reuse;
  HIP(hipEventCreateWithFlags(&reuse, hipEventDisableTiming));

  version_t *versions = (version_t *)xmalloc(sizeof(version_t) * (n_steps + 1));
  uint8_t *mask = (uint8_t *)xmalloc(N);
  memset(mask, 1, N);
  versions[0] = pack_version(c, t_base, mask, N, rec);
  LC(lc_store_append_async(store, t_base, mask, versions[0].payload, versions[0].bytes, stream, reuse));

  double *u = (double *)xmalloc(8 * N), *delta = (double *)xmalloc(8 * N);
  double *u_static = (double *)xmalloc(8 * N), *d_u_static = NULL;
  HIP(hipMalloc((void **)&d_u_static, 8 * N));
  int64_t *t_last = (int64_t *)xmalloc(8 * N);
  for (uint32_t k = 1; k <= n_steps; ++k) {
    const int64_t t = t_base + k;
    LOAD_STATE();
    /* the allocation-free score of the same weights and shadow, before the
     * context's pass (which refreshes the shadow in ACCUM mode): the same u,
     * bit for bit */
    LC(lc_score_layers_static(segs, S, N, (int32_t)dtype, eps_w, d_u_static, stream));
    HIP(hipMemcpy(u_static, d_u_static, 8 * N, hipMemcpyDeviceToHost));
    LC(lc_score_layers(c, t));
    lc_select_stats st;
    LC(lc_select(c, t, lr_scale[k], mask, &st));
    LC(lc_read_state(c, u, delta, t_last));
    if (memcmp(u, u_static, 8 * N) != 0) die("lc_score_layers_static disagrees with lc_score_layers");
    wr(u, 8 * N);
    wr(delta, 8 * N);
    wr(t_last, 8 * N);
    wr(mask, N);
    wr(&st.n_selected, 4);
    wr(&st.n_forced, 4);
    wr(&st.payload_bytes, 8);
    wr(&st.max_age, 8);
    wr(&st.weighted_age, 8);
    versions[k] = pack_version(c, t, mask, N, rec);
    LC(lc_store_append_async(store, t, mask, versions[k].payload, versions[k].bytes, stream, reuse));
  }

  /* fail-stop: the live state is lost, then rebuilt from the versions */
  HIP(hipMemset(dW, 0, total * esz));
  HIP(hipMemset(dS, 0, total * esz));
  if (has_master) HIP(hipMemset(dM, 0, total * 4));
  HIP(hipMemset(dm, 0, total * 4));
  HIP(hipMemset(dv, 0, total * 4));
  HIP(hipDeviceSynchronize());
  lc_version *lv = (lc_version *)xmalloc(sizeof(lc_version) * (n_steps + 1));
  for (uint32_t k = 0; k <= n_steps; ++k) {
    lv[k].step = versions[k].step;
    lv[k].mask = versions[k].mask;
    lv[k].payload = versions[k].payload;
    lv[k].payload_bytes = versions[k].bytes;
  }
  int64_t *chosen = (int64_t *)xmalloc(8 * N);
  LC(lc_restore_composite(c, lv, n_steps + 1, t_fail, chosen));
  LC(lc_read_state(c, NULL, NULL, t_last));
  wr(chosen, 8 * N);
  wr(t_last, 8 * N);
  uint8_t *rW = snapshot(dW, total * esz), *rS = snapshot(dS, total * esz);
  uint8_t *rM = has_master ? snapshot(dM, total * 4) : NULL;
  uint8_t *rm = snapshot(dm, total * 4), *rv = snapshot(dv, total * 4);
  wr(rW, total * esz);
  wr(rS, total * esz);
  if (has_master) wr(rM, total * 4);
  wr(rm, total * 4);
  wr(rv, total * 4);

  /* the same recovery from the store's files */
  LC(lc_store_sync(store));
  uint32_t n_stored = 0;
  LC(lc_store_count(store, &n_stored));
  if (n_stored != n_steps + 1) die("the store should hold every appended version");
  int64_t *planned = (int64_t *)xmalloc(8 * N);
  LC(lc_store_plan(store, t_fail, planned));
  if (memcmp(planned, chosen, 8 * N)) die("the store's plan differs from the composite restore's");
  HIP(hipMemset(dW, 0, total * esz));
  HIP(hipMemset(dS, 0, total * esz));
  if (has_master) HIP(hipMemset(dM, 0, total * 4));
  HIP(hipMemset(dm, 0, total * 4));
  HIP(hipMemset(dv, 0, total * 4));
  HIP(hipDeviceSynchronize());
  LC(lc_store_restore(store, c, t_fail, planned));
  uint8_t *h = (uint8_t *)xmalloc(total * 4);
#define SAME(dev, ref, n, what)                                   \
  do {                                                            \
    HIP(hipMemcpy(h, dev, n, hipMemcpyDeviceToHost));             \
    if (memcmp(h, ref, n)) die("restore from the store: " what);  \
  } while (0)
  SAME(dW, rW, total * esz, "weights differ");
  SAME(dS, rS, total * esz, "shadow differs");
  if (has_master) SAME(dM, rM, total * 4, "master differs");
  SAME(dm, rm, total * 4, "m differs");
  SAME(dv, rv, total * 4, "v differs");
  LC(lc_store_close(store));
  HIP(hipEventDestroy(reuse));

  /* an error path through the interface: a restore before any version */
  if (lc_restore_composite(c, lv, n_steps + 1, t_base - 1, NULL) != LC_ERR_NO_VERSION)
    die("a restore before the base should report LC_ERR_NO_VERSION");
  if (strlen(lc_last_error()) == 0) die("lc_last_error should describe the failure");

  LC(lc_destroy(c));
  for (uint32_t k = 0; k <= n_steps; ++k) {
    if (versions[k].payload) HIP(hipFree(versions[k].payload));
    free(versions[k].mask);
  }
  HIP(hipFree(d_u_static));
  free(u_static);
  HIP(hipFree(dW));
  HIP(hipFree(dS));
  if (dM) HIP(hipFree(dM));
  HIP(hipFree(dm));
  HIP(hipFree(dv));
  HIP(hipStreamDestroy(stream));
  if (fclose(out_f) != 0) die("closing the output failed");
  fclose(in);
  return 0;
}
