// C ABI entry points of libopattr: argument checks, workspace plan, stage
// sequencing on the caller's stream.
#include <string.h>

#include <mutex>

#include "accum.h"
#include "common.h"
#include "impl.h"

namespace opa {

static size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

struct Bump {
  size_t off = 0;
  size_t take(size_t bytes) {
    const size_t o = off;
    off = align_up(off + (bytes ? bytes : 1));
    return o;
  }
};

static bool has_dedup(const opattr_kernels *k, const opattr_dims *d) {
  return k && k->part_id && d->part_rep && d->n_parts > 0;
}

Plan make_plan(const opattr_kernels *k, const opattr_profiled *p, const opattr_ranges *r,
               const opattr_dims *d, bool second_match) {
  Plan pl{};
  pl.T = k ? k->n : 0;
  pl.P = p ? p->n : 0;
  pl.R = r ? r->n : 0;
  pl.NN = d->n_names;
  pl.NS = d->n_streams;
  pl.G = d->n_ops + 1;
  pl.NP = d->n_parts;
  pl.seq_dense = (d->flags & OPATTR_SEQ_DENSE) != 0;
  pl.ranges_nested = (d->flags & OPATTR_RANGES_NESTED) != 0;
  // seq tiles straight from per-stream segments: needs both kernel promises,
  // a matching stage (profiled rows given) and few streams and names (under
  // OPATTR_VALIDATE both promises are checked beside it: the layout by
  // check_kernel_layout, the density by the launch-order view's scatter)
  const bool seg_ok = pl.seq_dense && p != nullptr && pl.NS >= 1 && pl.NS <= 64 &&
                      pl.NN <= kFastNames;
  const bool sm_hint = (d->flags & OPATTR_KERNELS_STREAM_MAJOR) != 0;
  // dense seq in another order: opattr_attribute permutes the launches into
  // stream-major order when the fused path would then take them (not under
  // OPATTR_VALIDATE, which checks the caller's layout as given)
  const bool remap_ok = !sm_hint && seg_ok && !(d->flags & OPATTR_VALIDATE) && !second_match &&
                        r != nullptr && pl.G <= kFusedMaxRows && pl.R * 16 <= pl.T && pl.T > 0;
  pl.seg = (sm_hint || remap_ok) && seg_ok;  // sizes; reset below for the remapped case
  pl.nt = (pl.T + OPA_TILE - 1) / OPA_TILE;
  pl.ntp = (pl.P + OPA_TILE - 1) / OPA_TILE;
  pl.ncht = (pl.nt + kColChunk - 1) / kColChunk;
  pl.nchp = (pl.ntp + kColChunk - 1) / kColChunk;
  pl.ntr_max = pl.R / kRangeTile + (int64_t)pl.NS + 1;
  pl.nencb = (pl.T + kEncSpan - 1) / kEncSpan;
  pl.ntrt = (pl.T + OPA_TILE - 1) / OPA_TILE;
  pl.nchr = (pl.ntrt + kColChunk - 1) / kColChunk;
  const bool dd = has_dedup(k, d);
  const size_t T = (size_t)pl.T, P = (size_t)pl.P, R = (size_t)pl.R, NN = pl.NN;
  Bump b;
  // the launch-order view: unused on the segment path, but the standalone
  // dedup (no profiled rows, so never the segment path) needs it, and the
  // size for all inputs must cover every entry point
  pl.sv = b.take(T * 4);
  pl.kblk = b.take(pl.seg ? ((size_t)pl.NS + 2) * 8 : 0);
  pl.tbnd = b.take(pl.seg ? ((size_t)pl.nt + 1) * pl.NS * 4 : 0);
  pl.rk = b.take(pl.seq_dense ? 0 : T * 4);
  pl.seqsort_k0 = b.take(pl.seq_dense ? 0 : T * 4);
  pl.seqsort_k1 = b.take(pl.seq_dense ? 0 : T * 4);
  pl.seqsort_v0 = b.take(pl.seq_dense ? 0 : T * 4);
  pl.seqsort_v1 = b.take(pl.seq_dense ? 0 : T * 4);
  // radix histograms of the seq sort
  pl.rs_hist = b.take(radix_hist_entries(pl.seq_dense ? 0 : pl.T) * 4);
  pl.tlh = b.take((size_t)pl.nt * NN * 4);
  pl.pfh = b.take((size_t)pl.ntp * NN * 4);
  pl.tlch = b.take((size_t)pl.ncht * NN * 4);
  pl.pfch = b.take((size_t)pl.nchp * NN * 4);
  pl.tlc = b.take(NN * 4);
  pl.pfc = b.take(NN * 4);
  pl.off = b.take(NN * 4);
  pl.slot = b.take(P * 4);
  pl.pfirst = b.take(dd ? (size_t)pl.NP * 4 : 0);
  pl.plast = b.take(dd ? (size_t)pl.NP * 4 : 0);
  pl.pheads = b.take(dd ? (size_t)pl.NP * 4 : 0);
  pl.prec = b.take(dd ? (size_t)pl.NP * 8 : 0);
  pl.mbs = b.take(dd || pl.seg ? T * 4 : 0);
  pl.nbs = b.take(T * 4);  // dedup source names, or the fast path's key and in-tile rank
  pl.bcnt = b.take(pl.seg ? (size_t)pl.nt * 4 : 0);
  // the fused attribution keeps one partial result per run of launches of
  // one operator row; ranges at most one per 16 launches keep the runs long
  // enough for its per-block capacity (the rest would go through atomics)
  // (only opattr_attribute, which always has ranges, takes it: a plan
  // without ranges must stay within the size of the plan with them)
  pl.fused = pl.seg && r != nullptr && pl.G <= kFusedMaxRows && pl.R * 16 <= pl.T && pl.T > 0;
  pl.acc = b.take(pl.fused ? fused_acc_bytes(pl.G) : 0);
  pl.fbkt = b.take(pl.fused ? fused_bkt_bytes(pl.T) : 0);
  pl.forder = b.take(pl.fused ? (size_t)fused_agg_blocks(pl.T) * 4 : 0);
  pl.fsplit = b.take(pl.fused ? fused_split_bytes(pl.G) : 0);
  pl.fhot = b.take(pl.fused ? fused_hot_bytes() : 0);
  const bool rs = !pl.ranges_nested;
  pl.rperm = b.take(rs ? R * 4 : 0);
  pl.rs_c = b.take(rs ? R * 8 : 0);
  pl.re_c = b.take(rs ? R * 8 : 0);
  pl.rst_c = b.take(rs ? R * 2 : 0);
  pl.rop_c = b.take(rs ? R * 4 : 0);
  pl.rkd_c = b.take(rs && r && r->kind ? R : 0);
  pl.rsort_k0 = b.take(rs ? R * 8 : 0);
  pl.rsort_k1 = b.take(rs ? R * 8 : 0);
  pl.rsort_v0 = b.take(rs ? R * 4 : 0);
  pl.rsort_st = b.take(rs ? R * 2 : 0);
  pl.ree = b.take(R * 8);
  pl.npg = b.take(R * 4);
  pl.mxv = b.take(R * 8);
  pl.wfirst = b.take(R * 4);
  pl.wfused = b.take(R);
  pl.rblk = b.take(((size_t)pl.NS + 1) * 8);
  pl.tbase = b.take(((size_t)pl.NS + 1) * 4);
  const size_t ntr = (size_t)pl.ntr_max;
  pl.tM = b.take(ntr * 8);
  pl.tnpg = b.take(ntr * 4);
  pl.tnpg2 = b.take(ntr * 4);
  pl.tmx = b.take(ntr * 8);
  pl.tmx2 = b.take(ntr * 8);
  pl.tfirst = b.take(ntr * 4);
  pl.tlast = b.take(ntr * 4);
  pl.sflag = b.take((size_t)sflag_words(pl.NS) * 4);
  // aggregation: items (at most one per launch), partial rows (at most
  // kEncRowsPerWave per 64 * 8 launches), windows of 64 sorted items
  pl.cap_items = pl.T;
  pl.cap_rows = pl.nencb * (kEncThreads / OPA_WAVE) * kEncRowsPerWave;
  pl.max_windows = pl.cap_items / 64 + 1;
  pl.wi = b.take((size_t)pl.nencb * (kEncThreads / OPA_WAVE) * 4);
  pl.wr = b.take((size_t)pl.nencb * (kEncThreads / OPA_WAVE) * 4);
  pl.hmb = b.take((size_t)pl.nencb * kEncThreads);
  pl.ig = b.take((size_t)pl.cap_items * 4);
  pl.ia = b.take((size_t)pl.cap_items * 4);
  pl.ib = b.take((size_t)pl.cap_items * 4);
  pl.rows = b.take((size_t)pl.cap_rows * 200);
  pl.fparts = pl.rows;  // the fused attribution's kept partials (never both in one call)
  pl.meta = b.take(8 * 8);
  // item sort: per-tile row histograms for few rows, else one radix sort
  const bool few_rows = pl.G <= kFastKeys;
  pl.ith = b.take(few_rows ? (size_t)pl.ntrt * pl.G * 4 : 0);
  pl.itch = b.take(few_rows ? (size_t)pl.nchr * pl.G * 4 : 0);
  const size_t ni = few_rows ? 0 : (size_t)pl.cap_items;
  pl.isort_k0 = b.take(ni * 4);
  pl.isort_k1 = b.take(ni * 4);
  pl.isort_v0 = b.take(ni * 4);
  pl.isort_v1 = b.take(ni * 4);
  pl.isort_hist = b.take(few_rows ? 0 : radix_hist_entries((int64_t)ni) * 4);
  pl.gcnt = b.take((size_t)pl.G * 4);
  pl.goff = b.take(((size_t)pl.G + 1) * 4);
  // heavy rows (over 256 windows of 64 items, so at most items / 16320 of
  // them) as (row, first chunk) pairs, and their chunks of 256 windows: at
  // most about items / 8000, below max_windows / 64
  pl.heavy = b.take((size_t)pl.G * 8);
  pl.hcap = pl.max_windows / 64 + 64;
  pl.hch = b.take((size_t)pl.hcap * 8);
  pl.hpart = b.take((size_t)pl.hcap * 200);
  pl.multi = b.take((size_t)pl.G * 4);
  pl.sit = b.take((size_t)pl.cap_items * 8);
  pl.part = b.take((size_t)pl.max_windows * 2 * 200);
  // class discovery: per partition, and the key table
  const size_t NPc = d->n_parts, TS = (size_t)class_table_slots(d->n_parts);
  pl.c_first = b.take(NPc * 4);
  pl.c_last = b.take(NPc * 4);
  pl.c_runs = b.take(NPc * 4);
  pl.c_key = b.take(NPc * 8);
  pl.c_cand = b.take(NPc * 4);
  pl.c_fail = b.take(NPc * 4);
  pl.c_list = b.take(NPc * 4);
  pl.c_tkey = b.take(TS * 8);
  pl.c_tmin = b.take(TS * 4);
  pl.ident = b.take((size_t)d->n_ops * 4);
  pl.sumpart = b.take((size_t)kSumBlocks * 4 * 8);
  pl.misc = b.take(256);
  // a second set of the segment path's matching arrays, so that a second
  // matching (the tiered call's correlation lookup) can run beside the first
  pl.m2 = second_match && pl.seg;
  if (pl.m2) {
    pl.kblk2 = b.take(((size_t)pl.NS + 2) * 8);
    pl.tbnd2 = b.take(((size_t)pl.nt + 1) * pl.NS * 4);
    pl.tlh2 = b.take((size_t)pl.nt * NN * 4);
    pl.pfh2 = b.take((size_t)pl.ntp * NN * 4);
    pl.tlch2 = b.take((size_t)pl.ncht * NN * 4);
    pl.pfch2 = b.take((size_t)pl.nchp * NN * 4);
    pl.tlc2 = b.take(NN * 4);
    pl.pfc2 = b.take(NN * 4);
    pl.off2 = b.take(NN * 4);
    pl.slot2 = b.take(P * 4);
    pl.nbs2 = b.take(T * 4);
  }
  pl.remap = remap_ok && pl.fused;
  if (pl.remap) {
    pl.rm_hist = b.take(remap_hist_entries(pl) * 4);
    pl.rm_perm = b.take(T * 4);
    pl.rm_inv = b.take(T * 4);
    pl.rm_seq = b.take(T * 4);
    pl.rm_name = b.take(T * 4);
    pl.rm_dur = b.take(T * 4);
    pl.rm_st = b.take(T * 2);
    pl.rm_start = b.take(T * 8);
    pl.rm_query = b.take(k->query_ns ? T * 8 : 0);
    pl.rm_part = b.take(k->part_id ? T * 4 : 0);
    pl.rm_match = b.take(T * 4);
    pl.rm_rid = b.take(T * 4);
  }
  if (!sm_hint) pl.seg = pl.fused = false;  // the launches as given
  pl.total = b.off;
  return pl;
}

// the workspace regions are 256-byte aligned offsets from ws (vector loads)
static bool ws_ok(const void *ws, size_t ws_bytes, const Plan &pl) {
  return ws && (reinterpret_cast<uintptr_t>(ws) & 255) == 0 && ws_bytes >= pl.total;
}

// the summary's four sums over a stretch of table rows, per block
__global__ void __launch_bounds__(256) k_summary_part(const opattr_op_row *table, uint32_t G,
                                                      uint32_t NOPS, unsigned long long *part) {
  __shared__ unsigned long long red[4][4];
  unsigned long long at_ = 0, un = 0, tot = 0, mt = 0;
  for (uint32_t g = blockIdx.x * blockDim.x + threadIdx.x; g < G; g += gridDim.x * blockDim.x) {
    const unsigned long long t = table[g].total_ns;
    tot += t;
    mt += table[g].matched_ns;
    if (g < NOPS) at_ += t;
    else un += t;
  }
  at_ = wave_reduce_add(at_);
  un = wave_reduce_add(un);
  tot = wave_reduce_add(tot);
  mt = wave_reduce_add(mt);
  if (lane_id() == 0) {
    red[0][wave_id()] = at_;
    red[1][wave_id()] = un;
    red[2][wave_id()] = tot;
    red[3][wave_id()] = mt;
  }
  __syncthreads();
  if (threadIdx.x < 4)
    part[blockIdx.x * 4 + threadIdx.x] =
        red[threadIdx.x][0] + red[threadIdx.x][1] + red[threadIdx.x][2] + red[threadIdx.x][3];
}

// the finalisation by one block (body in common.h)
__global__ void __launch_bounds__(1024) k_finish(opattr_diag *diag, const uint8_t *sflag,
                                                 uint32_t ns, const unsigned long long *part,
                                                 int nparts, opattr_summary *sum) {
  finish_block(diag, sflag, ns, part, nparts, sum);
}

void launch_finish(opattr_diag *diag, const uint8_t *sflag, uint32_t ns, hipStream_t s,
                   const opattr_op_row *table, opattr_summary *sum, uint32_t G, uint32_t NOPS,
                   unsigned long long *part, int prepart) {
  probe_begin(OPATTR_PROBE_FINALIZE, s);
  int nb = prepart;
  if (table && prepart <= 0) {
    const uint32_t want = (G + 255) / 256;
    nb = (int)(want < (uint32_t)kSumBlocks ? (want > 0 ? want : 1) : kSumBlocks);
    k_summary_part<<<nb, 256, 0, s>>>(table, G, NOPS, part);
  }
  k_finish<<<1, 1024, 0, s>>>(diag, sflag, ns, table ? part : nullptr, nb, sum);
  probe_end(OPATTR_PROBE_FINALIZE, s);
}

static constexpr uint8_t kDefaultKind[OPATTR_NUM_COUNTERS] = {
    // counter appendix table, rows 1..20: SUM for additive counts, DW-mean for
    // rates and utilisations, MAX for per-kernel constants
    OPATTR_AGG_SUM,    OPATTR_AGG_SUM,    OPATTR_AGG_SUM,    OPATTR_AGG_DWMEAN,
    OPATTR_AGG_DWMEAN, OPATTR_AGG_DWMEAN, OPATTR_AGG_DWMEAN, OPATTR_AGG_DWMEAN,
    OPATTR_AGG_DWMEAN, OPATTR_AGG_DWMEAN, OPATTR_AGG_SUM,    OPATTR_AGG_DWMEAN,
    OPATTR_AGG_DWMEAN, OPATTR_AGG_DWMEAN, OPATTR_AGG_SUM,    OPATTR_AGG_DWMEAN,
    OPATTR_AGG_DWMEAN, OPATTR_AGG_MAX,    OPATTR_AGG_SUM,    OPATTR_AGG_MAX};

constexpr uint32_t kind_mask(uint8_t kind) {
  uint32_t m = 0;
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c)
    if (kDefaultKind[c] == kind) m |= 1u << c;
  return m;
}
static_assert(kind_mask(OPATTR_AGG_MAX) == kDefMaxMask && kind_mask(OPATTR_AGG_DWMEAN) == kDefDwMask,
              "default kinds and their masks disagree");

static const int64_t kMaxN = (int64_t)1 << 31;

static bool ok_n(int64_t n) { return n >= 0 && n < kMaxN; }

static bool check_dims(const opattr_dims *d) {
  if (!d) return false;
  if (d->n_names > kMaxNames) return false;
  if (d->n_streams > 65536u) return false;
  if (d->n_ops > kMaxOps || d->n_parts >= 0x7FFFFFFFu) return false;
  if (d->flags & ~(OPATTR_KERNELS_STREAM_MAJOR | OPATTR_SEQ_DENSE | OPATTR_RANGES_NESTED |
                   OPATTR_VALIDATE))
    return false;
  return true;
}

static bool check_kernels(const opattr_kernels *k, bool need_match, bool need_enc,
                          bool need_agg) {
  if (!k || !ok_n(k->n)) return false;
  if (k->n == 0) return true;
  if (need_match && (!k->seq || !k->name_id)) return false;
  if (need_enc && (!k->stream_id || !(k->query_ns || k->start_ns))) return false;
  if (need_agg && !k->dur_ns) return false;
  return true;
}

static bool check_profiled(const opattr_profiled *p, bool need_names, bool need_counters) {
  if (!p || !ok_n(p->n)) return false;
  if (p->n == 0) return true;
  if (need_names && !p->name_id) return false;
  if (need_counters && (!p->counters || p->row_stride < 0 || p->col_stride < 0)) return false;
  return true;
}

static bool check_ranges(const opattr_ranges *r) {
  if (!r || !ok_n(r->n)) return false;
  if (r->n == 0) return true;
  return r->start_ns && r->end_ns && r->stream_id && r->op_id;
}

// A side stream per device and calling thread (default priority), with the
// two events that fork work onto it from the caller's stream and join it
// back. NULL when it cannot be created; the caller's stream is used alone.
struct SideStream {
  hipStream_t s = nullptr, s2 = nullptr;
  hipEvent_t fork = nullptr, join = nullptr, fork2 = nullptr, join2 = nullptr,
             join3 = nullptr;
};
constexpr int kMaxDevices = 64;
inline thread_local SideStream g_side[kMaxDevices];

static SideStream *side_stream() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  SideStream &ss = g_side[dev];
  if (!ss.s) {
    SideStream n;
    bool ok = hipStreamCreateWithFlags(&n.s, hipStreamNonBlocking) == hipSuccess &&
              hipStreamCreateWithFlags(&n.s2, hipStreamNonBlocking) == hipSuccess;
    for (hipEvent_t *e : {&n.fork, &n.join, &n.fork2, &n.join2, &n.join3})
      ok = ok && hipEventCreateWithFlags(e, hipEventDisableTiming) == hipSuccess;
    if (!ok) {
      for (hipEvent_t e : {n.fork, n.join, n.fork2, n.join2, n.join3})
        if (e) (void)hipEventDestroy(e);
      for (hipStream_t t : {n.s, n.s2})
        if (t) (void)hipStreamDestroy(t);
      return nullptr;
    }
    ss = n;
  }
  return &ss;
}

// Library-held workspace of opattr_attribute_noalloc: every device that
// runs it holds its own copy until the process ends. In host code the
// array's name stands for no device address: scratch_ptr() gives this
// device's copy, taken once per device with that device current.
static __device__ __align__(256) uint8_t scratch[OPATTR_NOALLOC_SCRATCH_BYTES];
static void *g_scratch[kMaxDevices];
static std::mutex g_scratch_mu;

static void *scratch_ptr() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void *ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    g_scratch[dev] = ptr;
  }
  return g_scratch[dev];
}

static int launch_status() {
  const hipError_t launch = hipGetLastError();
  const hipError_t first = g_hip_error;
  g_hip_error = hipSuccess;
  return (launch == hipSuccess && first == hipSuccess) ? OPATTR_OK : OPATTR_ERR_HIP;
}

}  // namespace opa

using namespace opa;

extern "C" {

size_t opattr_workspace_bytes(const opattr_kernels *k, const opattr_profiled *p,
                              const opattr_ranges *r, const opattr_dims *d) {
  if (!d) return 0;
  return make_plan(k, p, r, d).total;
}

int opattr_diag_clear(opattr_diag *diag, void *stream) {
  if (!diag) return OPATTR_ERR_INVALID_ARG;
  fill_u32(reinterpret_cast<uint32_t *>(diag), 0, sizeof(opattr_diag) / 4, (hipStream_t)stream);
  return launch_status();
}

int opattr_read_diag(const opattr_diag *diag, opattr_diag *host_out, void *stream) {
  if (!diag || !host_out) return OPATTR_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  if (hipMemcpyAsync(host_out, diag, sizeof(opattr_diag), hipMemcpyDeviceToHost, s) != hipSuccess)
    return OPATTR_ERR_HIP;
  if (hipStreamSynchronize(s) != hipSuccess) return OPATTR_ERR_HIP;
  return OPATTR_OK;
}

int opattr_match(const opattr_kernels *k, const opattr_profiled *p, const opattr_dims *d,
                 int policy, int32_t *match, uint32_t *name_counts, opattr_diag *diag, void *ws,
                 size_t ws_bytes, void *stream) {
  if (!check_dims(d) || !check_kernels(k, true, false, false) || !check_profiled(p, true, false) ||
      !diag || policy < 0 || policy > 2 || (k->n > 0 && !match))
    return OPATTR_ERR_INVALID_ARG;
  const Plan pl = make_plan(k, p, nullptr, d);
  if (!ws_ok(ws, ws_bytes, pl)) return OPATTR_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  check_kernel_layout(k, d, diag, s);
  const bool validate = (d->flags & OPATTR_VALIDATE) != 0;
  build_seq_view(k, d, ws, pl, diag, validate, s);
  IomArgs a{k, p, d, policy, match, name_counts, diag, ws, &pl, false, validate};
  run_match(a, s);
  launch_finish(diag, nullptr, 0, s);
  return launch_status();
}

int opattr_dedup_broadcast(const opattr_kernels *k, const opattr_dims *d, int32_t *match,
                           const opattr_profiled *p, float *counters_out, opattr_diag *diag,
                           void *ws, size_t ws_bytes, void *stream) {
  if (!check_dims(d) || !check_kernels(k, true, false, false) || !diag ||
      (k->n > 0 && !match) || (counters_out && !check_profiled(p, false, true)))
    return OPATTR_ERR_INVALID_ARG;
  const Plan pl = make_plan(k, nullptr, nullptr, d);
  if (!ws_ok(ws, ws_bytes, pl)) return OPATTR_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  check_kernel_layout(k, d, diag, s);
  if (has_dedup(k, d)) {
    build_seq_view(k, d, ws, pl, diag, (d->flags & OPATTR_VALIDATE) != 0, s);
    run_dedup(k, d, match, diag, ws, pl, s);
  }
  if (counters_out) run_counters_out(p, match, k->n, counters_out, s);
  launch_finish(diag, nullptr, 0, s);
  return launch_status();
}

int opattr_dedup_classes(const opattr_kernels *k, const opattr_dims *d, int32_t *part_rep,
                         opattr_diag *diag, void *ws, size_t ws_bytes, void *stream) {
  if (!check_dims(d) || !k || !ok_n(k->n) || !diag || (d->n_parts > 0 && !part_rep) ||
      (k->n > 0 && (!k->seq || !k->name_id || !k->stream_id || !k->part_id)))
    return OPATTR_ERR_INVALID_ARG;
  const Plan pl = make_plan(k, nullptr, nullptr, d);
  if (!ws_ok(ws, ws_bytes, pl)) return OPATTR_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  check_kernel_layout(k, d, diag, s);
  if (d->n_parts > 0) {
    // the launch-order view: sorted when seq is not promised dense; a dense
    // seq is checked only under OPATTR_VALIDATE
    build_seq_view(k, d, ws, pl, diag, (d->flags & OPATTR_VALIDATE) != 0, s);
    run_classes(k, d, part_rep, diag, ws, pl, s);
  }
  launch_finish(diag, nullptr, 0, s);
  return launch_status();
}

int opattr_enclose_walk(const opattr_kernels *k, const opattr_ranges *r, const opattr_dims *d,
                        int32_t *range_id, uint8_t *fused, int32_t *range_any,
                        int32_t *range_parent, uint8_t *range_depth, opattr_diag *diag,
                        void *ws, size_t ws_bytes, void *stream) {
  if (!check_dims(d) || !check_kernels(k, false, true, false) || !check_ranges(r) || !diag ||
      (k->n > 0 && !range_id))
    return OPATTR_ERR_INVALID_ARG;
  const Plan pl = make_plan(k, nullptr, r, d);
  if (!ws_ok(ws, ws_bytes, pl)) return OPATTR_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  check_kernel_layout(k, d, diag, s);
  const bool validate = (d->flags & OPATTR_VALIDATE) != 0;
  const CoreRanges cr = prepare_ranges(r, d, ws, pl, diag, validate, s);
  resolve_ranges(cr, d, ws, pl, range_depth, diag, s, true);
  write_range_parents(cr, ws, pl, range_parent, s);
  EncArgs e{};
  e.k = k;
  e.cr = cr;
  e.d = d;
  e.range_id = range_id;
  e.fused = fused;
  e.range_any = range_any;
  e.diag = diag;
  e.ws = ws;
  e.pl = &pl;
  e.depth = true;
  e.range_depth = range_depth;
  run_enclose(e, s);
  launch_finish(diag, at<uint8_t>(ws, pl.sflag), d->n_streams, s);
  return launch_status();
}

int opattr_enclose_all(const opattr_kernels *k, const opattr_ranges *r, const opattr_dims *d,
                       int64_t *off, int32_t *ids, int64_t cap, opattr_diag *diag, void *ws,
                       size_t ws_bytes, void *stream) {
  if (!check_dims(d) || !check_kernels(k, false, true, false) || !check_ranges(r) || !diag ||
      !off || cap < 0 || (cap > 0 && !ids))
    return OPATTR_ERR_INVALID_ARG;
  const Plan pl = make_plan(k, nullptr, r, d);
  if (!ws_ok(ws, ws_bytes, pl)) return OPATTR_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  check_kernel_layout(k, d, diag, s);
  const CoreRanges cr = prepare_ranges(r, d, ws, pl, diag, (d->flags & OPATTR_VALIDATE) != 0, s);
  resolve_ranges(cr, d, ws, pl, nullptr, diag, s);
  run_enclose_all(cr, k, d, ws, pl, off, ids, cap, diag, s);
  launch_finish(diag, at<uint8_t>(ws, pl.sflag), d->n_streams, s);
  return launch_status();
}

int opattr_enclose(const opattr_kernels *k, const opattr_ranges *r, const opattr_dims *d,
                   int32_t *range_id, uint8_t *range_depth, opattr_diag *diag, void *ws,
                   size_t ws_bytes, void *stream) {
  return opattr_enclose_walk(k, r, d, range_id, nullptr, nullptr, nullptr, range_depth, diag, ws,
                             ws_bytes, stream);
}

static bool kinds_ok(const uint8_t *agg_kind) {
  if (!agg_kind) return true;
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c)
    if (agg_kind[c] > OPATTR_AGG_MAX) return false;
  return true;
}

int opattr_aggregate(const opattr_kernels *k, const opattr_profiled *p, const int32_t *match,
                     const int32_t *range_id, const opattr_ranges *r, const opattr_dims *d,
                     const uint8_t *agg_kind, opattr_op_row *table, opattr_summary *sum,
                     opattr_diag *diag, void *ws, size_t ws_bytes, void *stream) {
  if (!check_dims(d) || !check_kernels(k, false, false, true) || !check_profiled(p, false, true) ||
      !check_ranges(r) || !diag || !table || !sum || !kinds_ok(agg_kind) ||
      (k->n > 0 && (!match || !range_id)))
    return OPATTR_ERR_INVALID_ARG;
  const Plan pl = make_plan(k, p, r, d);
  if (!ws_ok(ws, ws_bytes, pl)) return OPATTR_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  check_kernel_layout(k, d, diag, s);
  EncArgs e{};
  e.k = k;
  e.p = p;
  e.match = match;
  e.r = r;
  e.d = d;
  e.range_id = const_cast<int32_t *>(range_id);
  e.agg_kind = agg_kind ? agg_kind : kDefaultKind;
  e.table = table;
  e.sum = sum;
  e.diag = diag;
  e.ws = ws;
  e.pl = &pl;
  run_aggregate_all(e, s);
  launch_finish(diag, nullptr, 0, s, table, sum, pl.G, d->n_ops,
                at<unsigned long long>(ws, pl.sumpart));
  return launch_status();
}

// opattr_attribute on the fused path (kernels stream-major with dense seq,
// ranges at most one per 16 launches): the ranges and the enclosure on a
// side stream, the profiled slot table on a second one, the matching up to
// the eligible launches' rows on the caller's stream; then one pass gives
// every launch its match (dedup broadcast included) and reduces the runs of
// launches of one operator row.
static int attribute_fused(const opattr_kernels *k, const opattr_profiled *p,
                           const opattr_ranges *r, const opattr_dims *d, int policy,
                           const uint8_t *agg_kind, int32_t *match, int32_t *range_id,
                           uint8_t *range_depth, uint32_t *name_counts, opattr_op_row *table,
                           opattr_summary *sum, opattr_diag *diag, void *ws, const Plan &pl,
                           hipStream_t s, bool fork, const opattr_kernels *k_given = nullptr) {
  SideStream *ss = fork ? side_stream() : nullptr;
  const hipStream_t s2 = ss ? ss->s : s;
  if (ss) {
    note(hipEventRecord(ss->fork, s));
    note(hipStreamWaitEvent(s2, ss->fork, 0));
  }
  const bool validate = (d->flags & OPATTR_VALIDATE) != 0;
  if (validate) {
    // the layout check goes first on the profiled rows' stream, whose work
    // ends before the other two streams' (the density of seq is checked in
    // the matching's tiles)
    const hipStream_t sc = ss ? ss->s2 : s;
    if (ss) note(hipStreamWaitEvent(sc, ss->fork, 0));
    check_kernel_layout(k, d, diag, sc);
  }
  FillJobs acc;  // the fused aggregation's accumulators, cleared with the ranges' state
  fused_acc_clear(acc, ws, pl);
  probe_begin(OPATTR_PROBE_RANGES, s2);
  const CoreRanges cr = prepare_ranges(r, d, ws, pl, diag, validate, s2, &acc);
  resolve_ranges(cr, d, ws, pl, range_depth, diag, s2, true);
  probe_end(OPATTR_PROBE_RANGES, s2);
  if (k_given) {
    // the launches given in another order: permuted (into k's arrays) on the
    // caller's stream while the ranges are sorted; the enclosure waits
    Plan pv = pl;
    pv.seg = false;  // the view is built here (the segment path reads none)
    build_seq_view(k_given, d, ws, pv, diag, false, s);
    remap_launches(k_given, d, ws, pl, nullptr, s);
    if (ss) {
      note(hipEventRecord(ss->join3, s));
      note(hipStreamWaitEvent(s2, ss->join3, 0));
    }
  }
  EncArgs e{};
  e.k = k;
  e.p = p;
  e.match = match;
  e.r = r;
  e.cr = cr;
  e.d = d;
  e.range_id = range_id;
  e.agg_kind = agg_kind ? agg_kind : kDefaultKind;
  e.table = table;
  e.sum = sum;
  e.diag = diag;
  e.ws = ws;
  e.pl = &pl;
  e.depth = true;
  e.range_depth = range_depth;
  run_enclose(e, s2);
  if (ss) note(hipEventRecord(ss->join, s2));
  IomArgs a{k, p, d, policy, match, name_counts, diag, ws, &pl, true, validate};
  a.buckets = true;
  a.fused_order = ss != nullptr;  // only where the profiled side has a stream of its own
  if (ss) {
    a.pf_stream = ss->s2;
    a.pf_fork = ss->fork2;
    a.pf_join = ss->join2;
  }
  run_match(a, s);
  const AggIn in = agg_inputs(e);
  FusedIn f{};
  f.k = k;
  f.r = r;
  f.d = d;
  f.range_id = range_id;
  f.match = match;
  f.in = &in;
  f.absent = p->absent_mask;
  f.table = table;
  f.diag = diag;
  f.ws = ws;
  f.pl = &pl;
  if (ss) note(hipStreamWaitEvent(s, ss->join, 0));
  f.sum = sum;
  f.ordered = a.fused_order;
  run_fused_agg(f, s);  // ends with the finalisation
  return launch_status();
}

static bool attribute_args_ok(const opattr_kernels *k, const opattr_profiled *p,
                              const opattr_ranges *r, const opattr_dims *d, int policy,
                              const uint8_t *agg_kind, int32_t *match, int32_t *range_id,
                              opattr_op_row *table, opattr_summary *sum, opattr_diag *diag) {
  return check_dims(d) && check_kernels(k, true, true, true) && check_profiled(p, true, true) &&
         check_ranges(r) && diag && table && sum && policy >= 0 && policy <= 2 &&
         kinds_ok(agg_kind) && (k->n == 0 || (match && range_id));
}

// opattr_attribute on dense seq given in another order: the launches
// permuted into stream-major order (through the launch-order view), the
// fused path on them, and the per-launch outputs permuted back.
static int attribute_remapped(const opattr_kernels *k, const opattr_profiled *p,
                              const opattr_ranges *r, const opattr_dims *d, int policy,
                              const uint8_t *agg_kind, int32_t *match, int32_t *range_id,
                              uint8_t *range_depth, uint32_t *name_counts, opattr_op_row *table,
                              opattr_summary *sum, opattr_diag *diag, void *ws, const Plan &pl,
                              hipStream_t s, bool fork) {
  opattr_kernels k2;
  remap_view(k, ws, pl, &k2);
  opattr_dims d2 = *d;
  d2.flags |= OPATTR_KERNELS_STREAM_MAJOR;
  Plan pf = pl;
  pf.seg = pf.fused = true;
  attribute_fused(&k2, p, r, &d2, policy, agg_kind, at<int32_t>(ws, pl.rm_match),
                  at<int32_t>(ws, pl.rm_rid), range_depth, name_counts, table, sum, diag, ws, pf,
                  s, fork, k);
  remap_back(ws, pl, match, range_id, s);
  return launch_status();
}

// The four stages on a checked plan and workspace; with fork, independent
// stages run on this thread's side streams, else all on the caller's stream.
static int attribute_call(const opattr_kernels *k, const opattr_profiled *p,
                          const opattr_ranges *r, const opattr_dims *d, int policy,
                          const uint8_t *agg_kind, int32_t *match, int32_t *range_id,
                          uint8_t *range_depth, uint32_t *name_counts, opattr_op_row *table,
                          opattr_summary *sum, opattr_diag *diag, void *ws, const Plan &pl,
                          hipStream_t s, bool fork) {
  if (pl.remap) return attribute_remapped(k, p, r, d, policy, agg_kind, match, range_id,
                                          range_depth, name_counts, table, sum, diag, ws, pl, s,
                                          fork);
  if (pl.fused) return attribute_fused(k, p, r, d, policy, agg_kind, match, range_id,
                                       range_depth, name_counts, table, sum, diag, ws, pl, s,
                                       fork);
  check_kernel_layout(k, d, diag, s);
  const bool validate = (d->flags & OPATTR_VALIDATE) != 0;
  // the ranges, the enclosure and the aggregation plan do not depend on the
  // matching: they run on a side stream of this device, joined back before
  // the run reduction (counts) and the per-row reduction (items)
  SideStream *ss = fork ? side_stream() : nullptr;
  const hipStream_t s2 = ss ? ss->s : s;
  if (ss) {
    note(hipEventRecord(ss->fork, s));
    note(hipStreamWaitEvent(s2, ss->fork, 0));
  }
  probe_begin(OPATTR_PROBE_RANGES, s2);
  const CoreRanges cr = prepare_ranges(r, d, ws, pl, diag, validate, s2);
  resolve_ranges(cr, d, ws, pl, range_depth, diag, s2);
  probe_end(OPATTR_PROBE_RANGES, s2);
  EncArgs e{};
  e.k = k;
  e.p = p;
  e.match = match;
  e.r = r;
  e.cr = cr;
  e.d = d;
  e.range_id = range_id;
  e.agg_kind = agg_kind ? agg_kind : kDefaultKind;
  e.table = table;
  e.sum = sum;
  e.diag = diag;
  e.ws = ws;
  e.pl = &pl;
  // the run reduction needs only the counts; the items and their sort
  // continue on the side stream beside the matching and the run reduction
  plan_counts(e, true, s2);
  if (ss) note(hipEventRecord(ss->join, s2));
  plan_emit(e, s2);
  triage_rows(e, s2);  // empty rows and the spread-row list, off the caller's path
  if (ss) note(hipEventRecord(ss->join3, s2));
  build_seq_view(k, d, ws, pl, diag, validate, s);
  IomArgs a{k, p, d, policy, match, name_counts, diag, ws, &pl, true, validate};
  if (ss) {
    a.pf_stream = ss->s2;
    a.pf_fork = ss->fork2;
    a.pf_join = ss->join2;
  }
  run_match(a, s);
  if (ss) note(hipStreamWaitEvent(s, ss->join, 0));
  reduce_runs(e, s);
  if (ss) note(hipStreamWaitEvent(s, ss->join3, 0));
  reduce_items(e, s, true);
  launch_finish(diag, at<uint8_t>(ws, pl.sflag), d->n_streams, s, table, sum, pl.G, d->n_ops,
                at<unsigned long long>(ws, pl.sumpart));
  return launch_status();
}

int opattr_attribute(const opattr_kernels *k, const opattr_profiled *p, const opattr_ranges *r,
                     const opattr_dims *d, int policy, const uint8_t *agg_kind, int32_t *match,
                     int32_t *range_id, uint8_t *range_depth, uint32_t *name_counts,
                     opattr_op_row *table, opattr_summary *sum, opattr_diag *diag, void *ws,
                     size_t ws_bytes, void *stream) {
  if (!attribute_args_ok(k, p, r, d, policy, agg_kind, match, range_id, table, sum, diag))
    return OPATTR_ERR_INVALID_ARG;
  const Plan pl = make_plan(k, p, r, d);
  if (!ws_ok(ws, ws_bytes, pl)) return OPATTR_ERR_WORKSPACE;
  return attribute_call(k, p, r, d, policy, agg_kind, match, range_id, range_depth, name_counts,
                        table, sum, diag, ws, pl, (hipStream_t)stream, true);
}

int opattr_attribute_noalloc(const opattr_kernels *k, const opattr_profiled *p,
                             const opattr_ranges *r, const opattr_dims *d, int policy,
                             const uint8_t *agg_kind, int32_t *match, int32_t *range_id,
                             uint8_t *range_depth, uint32_t *name_counts, opattr_op_row *table,
                             opattr_summary *sum, opattr_diag *diag, void *stream) {
  if (!attribute_args_ok(k, p, r, d, policy, agg_kind, match, range_id, table, sum, diag))
    return OPATTR_ERR_INVALID_ARG;
  const Plan pl = make_plan(k, p, r, d);
  if (pl.total > OPATTR_NOALLOC_SCRATCH_BYTES) return OPATTR_ERR_SCRATCH;
  void *ws = scratch_ptr();
  if (!ws) return OPATTR_ERR_HIP;
  return attribute_call(k, p, r, d, policy, agg_kind, match, range_id, range_depth, name_counts,
                        table, sum, diag, ws, pl, (hipStream_t)stream, false);
}

// the matching's view of a tiers call: the correlation entries as profiled
// rows, no partitions
struct TiersView {
  opattr_kernels k;
  opattr_profiled p;
  opattr_dims d;
  TiersView(const opattr_kernels *k0, const opattr_corr_map *corr, const opattr_dims *d0)
      : k(*k0), p{}, d(*d0) {
    k.part_id = nullptr;
    d.part_rep = nullptr;
    d.n_parts = 0;
    p.n = corr ? corr->n : 0;
    p.name_id = corr ? corr->name_id : nullptr;
  }
};

size_t opattr_tiers_workspace_bytes(const opattr_kernels *k, const opattr_corr_map *corr,
                                    const opattr_ranges *r, const opattr_dims *d) {
  if (!k || !d) return 0;
  const TiersView v(k, corr, d);
  return make_plan(&v.k, &v.p, r, &v.d).total;
}

int opattr_tiers(const opattr_kernels *k, const opattr_corr_map *corr,
                 const opattr_fusion_map *fmap, const opattr_ranges *r, const opattr_dims *d,
                 int corr_policy, const int32_t *range_id, const uint8_t *walk_fused,
                 uint8_t *tier, int32_t *op, uint8_t *fused, opattr_coverage *cov,
                 opattr_diag *diag, void *ws, size_t ws_bytes, void *stream) {
  if (!check_dims(d) || !k || !ok_n(k->n) || !r || !ok_n(r->n) || !diag || !cov ||
      corr_policy < 0 || corr_policy > 2)
    return OPATTR_ERR_INVALID_ARG;
  if (k->n > 0 && (!k->name_id || !k->dur_ns || !range_id || !tier || !op || !fused ||
                   (r->n > 0 && !r->op_id)))
    return OPATTR_ERR_INVALID_ARG;
  if (corr && (!ok_n(corr->n) || (corr->n > 0 && (!corr->name_id || !corr->op_id)) ||
               (k->n > 0 && !k->seq)))
    return OPATTR_ERR_INVALID_ARG;
  if (fmap && (!fmap->off || !fmap->op_id)) return OPATTR_ERR_INVALID_ARG;
  const TiersView v(k, corr, d);
  const Plan pl = make_plan(&v.k, &v.p, r, &v.d);
  if (!ws_ok(ws, ws_bytes, pl)) return OPATTR_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  const bool validate = (d->flags & OPATTR_VALIDATE) != 0;
  int32_t *entry = nullptr;
  if (corr) {
    // HIGH: Alg. 1 with the correlation entries as the rows
    check_kernel_layout(&v.k, &v.d, diag, s);
    entry = at<int32_t>(ws, pl.ia);
    build_seq_view(&v.k, &v.d, ws, pl, diag, validate, s);
    IomArgs a{&v.k, &v.p, &v.d, corr_policy, entry, nullptr, diag, ws, &pl, false, validate};
    run_match(a, s);
  }
  TierIn x{k, corr, fmap, r, d, entry, range_id, walk_fused, tier, op, fused, cov, diag, ws, &pl};
  run_tiers(x, s);
  launch_finish(diag, nullptr, 0, s);
  return launch_status();
}

// profiled rows sized for the larger of the profiled list and the map, so
// that one plan serves both matchings of the tiered call
static opattr_profiled tiered_rows(const opattr_profiled *p, const opattr_corr_map *corr) {
  opattr_profiled m = *p;
  if (corr && corr->n > m.n) m.n = corr->n;
  return m;
}

size_t opattr_attribute_tiered_workspace_bytes(const opattr_kernels *k, const opattr_profiled *p,
                                               const opattr_ranges *r,
                                               const opattr_corr_map *corr,
                                               const opattr_dims *d) {
  if (!k || !p || !d) return 0;
  const opattr_profiled m = tiered_rows(p, corr);
  return make_plan(k, &m, r, d, true).total;
}

// The plan with the segment path's matching arrays swapped for the second set.
static Plan second_match_plan(const Plan &pl) {
  Plan q = pl;
  if (!pl.m2) return q;
  q.kblk = pl.kblk2;
  q.tbnd = pl.tbnd2;
  q.tlh = pl.tlh2;
  q.pfh = pl.pfh2;
  q.tlch = pl.tlch2;
  q.pfch = pl.pfch2;
  q.tlc = pl.tlc2;
  q.pfc = pl.pfc2;
  q.off = pl.off2;
  q.slot = pl.slot2;
  q.nbs = pl.nbs2;
  return q;
}

int opattr_attribute_tiered(const opattr_kernels *k, const opattr_profiled *p,
                            const opattr_ranges *r, const opattr_corr_map *corr,
                            const opattr_fusion_map *fmap, const opattr_dims *d, int policy,
                            int corr_policy, const uint8_t *agg_kind, int32_t *match,
                            int32_t *range_id, uint8_t *tier, int32_t *op, uint8_t *fused,
                            opattr_op_row *table, opattr_summary *sum, opattr_coverage *cov,
                            opattr_diag *diag, void *ws, size_t ws_bytes, void *stream) {
  if (!check_dims(d) || !check_kernels(k, true, true, true) || !check_profiled(p, true, true) ||
      !check_ranges(r) || !diag || !table || !sum || !cov || policy < 0 || policy > 2 ||
      corr_policy < 0 || corr_policy > 2 || !kinds_ok(agg_kind) ||
      (k->n > 0 && (!match || !range_id || !tier || !op || !fused)))
    return OPATTR_ERR_INVALID_ARG;
  if (corr && (!ok_n(corr->n) || (corr->n > 0 && (!corr->name_id || !corr->op_id))))
    return OPATTR_ERR_INVALID_ARG;
  if (fmap && (!fmap->off || !fmap->op_id)) return OPATTR_ERR_INVALID_ARG;
  const opattr_profiled rows = tiered_rows(p, corr);
  const Plan pl = make_plan(k, &rows, r, d, true);
  if (!ws_ok(ws, ws_bytes, pl)) return OPATTR_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  check_kernel_layout(k, d, diag, s);
  const bool validate = (d->flags & OPATTR_VALIDATE) != 0;
  // the ranges and the walk need no match: a side stream, joined back
  // before the tiers
  SideStream *ss = side_stream();
  const hipStream_t s2 = ss ? ss->s : s;
  if (ss) {
    note(hipEventRecord(ss->fork, s));
    note(hipStreamWaitEvent(s2, ss->fork, 0));
  }
  probe_begin(OPATTR_PROBE_RANGES, s2);
  const CoreRanges cr = prepare_ranges(r, d, ws, pl, diag, validate, s2);
  resolve_ranges(cr, d, ws, pl, nullptr, diag, s2, true);
  probe_end(OPATTR_PROBE_RANGES, s2);
  EncArgs w{};
  w.k = k;
  w.cr = cr;
  w.d = d;
  w.range_id = range_id;
  w.fused = fused;
  w.diag = diag;
  w.ws = ws;
  w.pl = &pl;
  w.depth = true;
  run_enclose(w, s2);
  if (ss) note(hipEventRecord(ss->join, s2));
  // matching with the dedup broadcast, then the correlation lookup (Alg. 1
  // over the map's entries, partitions off) into the item array
  build_seq_view(k, d, ws, pl, diag, validate, s);
  // the correlation lookup needs only the launches and the map: on the
  // segment path it runs on the second side stream with its own arrays,
  // beside the matching of the profiled rows
  int32_t *entry = nullptr;
  const TiersView v(k, corr, d);
  const Plan pl2 = second_match_plan(pl);
  const bool beside = corr && ss && pl.m2;
  if (corr) {
    entry = at<int32_t>(ws, pl.ia);
    if (beside) {
      note(hipEventRecord(ss->fork2, s));
      note(hipStreamWaitEvent(ss->s2, ss->fork2, 0));
      IomArgs c{&v.k, &v.p, &v.d, corr_policy, entry, nullptr, diag, ws, &pl2, false, validate};
      run_match(c, ss->s2);
      note(hipEventRecord(ss->join2, ss->s2));
    }
  }
  IomArgs a{k, p, d, policy, match, nullptr, diag, ws, &pl, true, validate};
  run_match(a, s);
  if (corr && !beside) {
    IomArgs c{&v.k, &v.p, &v.d, corr_policy, entry, nullptr, diag, ws, &pl, false, validate};
    run_match(c, s);
  }
  if (beside) note(hipStreamWaitEvent(s, ss->join2, 0));
  if (ss) note(hipStreamWaitEvent(s, ss->join, 0));
  TierIn x{k, corr, fmap, r, d, entry, range_id, fused, tier, op, fused, cov, diag, ws, &pl};
  run_tiers(x, s);
  // the table by tier operator
  uint32_t *ident = at<uint32_t>(ws, pl.ident);
  launch_iota(ident, d->n_ops, s);
  opattr_ranges ops{};
  ops.n = d->n_ops;
  ops.op_id = ident;
  EncArgs e{};
  e.k = k;
  e.p = p;
  e.match = match;
  e.r = &ops;
  e.d = d;
  e.range_id = op;
  e.agg_kind = agg_kind ? agg_kind : kDefaultKind;
  e.table = table;
  e.sum = sum;
  e.diag = diag;
  e.ws = ws;
  e.pl = &pl;
  run_aggregate_all(e, s);
  launch_finish(diag, at<uint8_t>(ws, pl.sflag), d->n_streams, s, table, sum, pl.G, d->n_ops,
                at<unsigned long long>(ws, pl.sumpart));
  return launch_status();
}

int opattr_aggregate_ops(const opattr_kernels *k, const opattr_profiled *p, const int32_t *match,
                         const int32_t *op, const opattr_dims *d, const uint8_t *agg_kind,
                         opattr_op_row *table, opattr_summary *sum, opattr_diag *diag,
                         void *ws, size_t ws_bytes, void *stream) {
  if (!check_dims(d) || !check_kernels(k, false, false, true) || !check_profiled(p, false, true) ||
      !diag || !table || !sum || !kinds_ok(agg_kind) || (k->n > 0 && (!match || !op)))
    return OPATTR_ERR_INVALID_ARG;
  const Plan pl = make_plan(k, p, nullptr, d);
  if (!ws_ok(ws, ws_bytes, pl)) return OPATTR_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  // the operators stand in for range ids over the identity op table
  uint32_t *ident = at<uint32_t>(ws, pl.ident);
  launch_iota(ident, d->n_ops, s);
  opattr_ranges ops{};
  ops.n = d->n_ops;
  ops.op_id = ident;
  EncArgs e{};
  e.k = k;
  e.p = p;
  e.match = match;
  e.r = &ops;
  e.d = d;
  e.range_id = const_cast<int32_t *>(op);
  e.agg_kind = agg_kind ? agg_kind : kDefaultKind;
  e.table = table;
  e.sum = sum;
  e.diag = diag;
  e.ws = ws;
  e.pl = &pl;
  run_aggregate_all(e, s);
  launch_finish(diag, nullptr, 0, s, table, sum, pl.G, d->n_ops,
                at<unsigned long long>(ws, pl.sumpart));
  return launch_status();
}

// the aggregation's view of a per-dispatch call: R + n_ops operator rows
static opattr_dims dispatch_dims(const opattr_ranges *r, const opattr_dims *d) {
  opattr_dims dd = *d;
  dd.n_ops = (uint32_t)(r->n + d->n_ops);
  return dd;
}

size_t opattr_dispatch_workspace_bytes(const opattr_kernels *k, const opattr_profiled *p,
                                       const opattr_ranges *r, const opattr_dims *d) {
  if (!d || !r || r->n < 0 || r->n + (int64_t)d->n_ops > (int64_t)kMaxOps) return 0;
  const opattr_dims dd = dispatch_dims(r, d);
  return make_plan(k, p, nullptr, &dd).total;
}

int opattr_aggregate_dispatch(const opattr_kernels *k, const opattr_profiled *p,
                              const int32_t *match, const int32_t *range_id, const int32_t *op,
                              const opattr_ranges *r, const opattr_dims *d,
                              const uint8_t *agg_kind, opattr_op_row *table, opattr_summary *sum,
                              int32_t *row, opattr_diag *diag, void *ws, size_t ws_bytes,
                              void *stream) {
  if (!check_dims(d) || !check_kernels(k, false, false, true) || !check_profiled(p, false, true) ||
      !r || !ok_n(r->n) || r->n + (int64_t)d->n_ops > (int64_t)kMaxOps || !diag || !table ||
      !sum || !kinds_ok(agg_kind) || (k->n > 0 && (!match || !range_id)) ||
      (r->n > 0 && !r->op_id))
    return OPATTR_ERR_INVALID_ARG;
  const opattr_dims dd = dispatch_dims(r, d);
  const Plan pl = make_plan(k, p, nullptr, &dd);
  if (!ws_ok(ws, ws_bytes, pl)) return OPATTR_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  // per-launch rows in the launch-order view's space (unused here), then
  // the aggregation by those rows over an identity op table
  int32_t *key = at<int32_t>(ws, pl.sv);
  launch_dispatch_keys(range_id, op, r, d->n_ops, pl.T, key, row, diag, s);
  uint32_t *ident = at<uint32_t>(ws, pl.ident);
  launch_iota(ident, dd.n_ops, s);
  opattr_ranges rows{};
  rows.n = dd.n_ops;
  rows.op_id = ident;
  EncArgs e{};
  e.k = k;
  e.p = p;
  e.match = match;
  e.r = &rows;
  e.d = &dd;
  e.range_id = key;
  e.agg_kind = agg_kind ? agg_kind : kDefaultKind;
  e.table = table;
  e.sum = sum;
  e.diag = diag;
  e.ws = ws;
  e.pl = &pl;
  run_aggregate_all(e, s);
  launch_finish(diag, nullptr, 0, s, table, sum, pl.G, dd.n_ops,
                at<unsigned long long>(ws, pl.sumpart));
  return launch_status();
}

int opattr_set_class_key_bits(int bits) {
  if (bits < 1 || bits > 64) return OPATTR_ERR_INVALID_ARG;
  g_class_key_bits = bits;
  return OPATTR_OK;
}

int opattr_set_probe_events(void *const *events, int n) {
  if (n < 0 || n > OPATTR_NUM_PROBES || (n > 0 && !events)) return OPATTR_ERR_INVALID_ARG;
  g_probes.n = events ? n : 0;
  for (int i = 0; i < 2 * OPATTR_NUM_PROBES; ++i)
    g_probes.ev[i] = (events && i < 2 * n) ? (hipEvent_t)events[i] : nullptr;
  return OPATTR_OK;
}

const char *opattr_strerror(int status) {
  switch (status) {
    case OPATTR_OK: return "ok";
    case OPATTR_ERR_INVALID_ARG: return "invalid argument";
    case OPATTR_ERR_WORKSPACE: return "workspace too small";
    case OPATTR_ERR_HIP: return "HIP launch failed";
    case OPATTR_ERR_COUNT_MISMATCH: return "per-name invocation counts differ (strict policy)";
    case OPATTR_ERR_NOT_NESTED: return "ranges of a stream cross";
    case OPATTR_ERR_DEDUP: return "positional dedup lookup failed";
    case OPATTR_ERR_PARTITION: return "a partition is not one contiguous run of launches";
    case OPATTR_ERR_ORDER: return "launch order violated (duplicate seq or false layout promise)";
    case OPATTR_ERR_DATA: return "id out of range or malformed range";
    case OPATTR_ERR_LIMIT: return "range nesting deeper than 255";
    case OPATTR_ERR_SCRATCH: return "the call needs more than the library's scratch";
    default: return "unknown status";
  }
}

}  // extern "C"
