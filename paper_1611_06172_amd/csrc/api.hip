// C ABI of libw2v (declared in include/w2v.h): argument validation, error
// reporting and kernel launches. Every check runs on the host before any HIP
// call, so a rejected call has no device side effect.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>

#include "kernel_args.h"
#include "w2v_internal.h"

namespace w2v {

static thread_local char g_error[512] = "";

int fail(int code, const char* msg) {
  snprintf(g_error, sizeof(g_error), "%s", msg);
  return code;
}

int failf(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_error, sizeof(g_error), fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_error[0] = '\0';
  return W2V_OK;
}

static int hip_fail(hipError_t e, const char* what) {
  return failf(W2V_EHIP, "%s: %s", what, hipGetErrorString(e));
}

// Per-device state set up by w2v_init (or by the first GPU call on the
// device): the error word, one int32 of pinned host memory mapped into the
// device's address space. Kernels that skip a minibatch for an id outside
// [0, V) store kStatusBadId into it (a system-scope store, so the host reads
// it without a copy or a synchronisation); every later call on the device
// reports it once as W2V_EDEVICE_FLAG and clears it.
constexpr int kMaxDevices = 64;

struct DeviceState {
  bool ready = false;
  volatile int32_t* status_host = nullptr;  // what the host reads
  int32_t* status_dev = nullptr;            // the same word, device address
  void* scratch = nullptr;                  // this device's copy of `scratch`
};

static std::mutex g_dev_mu;
static DeviceState g_dev[kMaxDevices];

static int current_device(int& dev) {
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return failf(W2V_EUNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
  return W2V_OK;
}

// Scratch memory of w2v_train_epoch_noalloc: the split rows' partial rows,
// W2V_NOALLOC_SCRATCH_BYTES per device, held until the process ends. Host
// code never passes `scratch` itself to a kernel (in host code it names a
// host-side stand-in); it uses the device address hipGetSymbolAddress gives
// for the current device, recorded in DeviceState::scratch.
static __device__ __align__(256) unsigned char scratch[W2V_NOALLOC_SCRATCH_BYTES];

// Sets up the current device's state once (caller holds g_dev_mu).
static int setup_device_locked(int dev) {
  DeviceState& st = g_dev[dev];
  if (st.ready) return W2V_OK;
  void* sym = nullptr;
  hipError_t es = hipGetSymbolAddress(&sym, HIP_SYMBOL(scratch));
  if (es != hipSuccess) return hip_fail(es, "hipGetSymbolAddress of the scratch array");
  if (sym == nullptr || ((uintptr_t)sym & 255u) != 0)
    return fail(W2V_EHIP, "scratch array address is NULL or not 256-byte aligned");
  void* host = nullptr;
  hipError_t e = hipHostMalloc(&host, 256, hipHostMallocMapped | hipHostMallocCoherent);
  if (e != hipSuccess) return hip_fail(e, "hipHostMalloc of the error word");
  void* mapped = nullptr;
  e = hipHostGetDevicePointer(&mapped, host, 0);
  if (e != hipSuccess) {
    (void)hipHostFree(host);
    return hip_fail(e, "hipHostGetDevicePointer of the error word");
  }
  st.status_host = (volatile int32_t*)host;
  *st.status_host = 0;
  st.status_dev = (int32_t*)mapped;
  st.scratch = sym;
  st.ready = true;
  return W2V_OK;
}

// Entry check of every GPU call: sets up the device if needed (unless
// `no_setup`, for the entry point that must not allocate: it then fails
// when w2v_init has not run on the device), reports (and clears) a skip
// recorded by an earlier call, and gives the kernels the error word and
// the device's scratch address. A reported skip means this call launched
// nothing.
static int enter_device(int32_t** status_dev, void** scratch_dev = nullptr,
                        bool no_setup = false) {
  int dev = 0;
  int rc = current_device(dev);
  if (rc != W2V_OK) return rc;
  std::lock_guard<std::mutex> lock(g_dev_mu);
  if (no_setup && !g_dev[dev].ready)
    return failf(W2V_EINVAL,
                 "w2v_init has not run on device %d: the entry point that allocates "
                 "nothing needs it first",
                 dev);
  rc = setup_device_locked(dev);
  if (rc != W2V_OK) return rc;
  DeviceState& st = g_dev[dev];
  if (scratch_dev != nullptr) *scratch_dev = st.scratch;
  if (*st.status_host != 0) {
    *st.status_host = 0;
    return failf(W2V_EDEVICE_FLAG,
                 "an earlier call on device %d skipped work: an id outside [0, V) "
                 "in the corpus, the negative table or a batch (stats[3] counts them); "
                 "this call launched nothing",
                 dev);
  }
  *status_dev = st.status_dev;
  return W2V_OK;
}

// Compute units of the current device (queried once per device).
static int cu_count() {
  static std::mutex mu;
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  std::lock_guard<std::mutex> lock(mu);
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) ==
        hipSuccess)
      cached[dev] = n;
  }
  return cached[dev];
}

struct SamplingCheck {
  const int32_t* corpus;
  int64_t T, pos_begin, pos_end;
  int32_t L, V, window, K;
  const int32_t* table;
  int64_t table_size;
  int32_t epoch, n_epochs;
};

static int check_sampling(const SamplingCheck& c) {
  if (c.corpus == nullptr) return fail(W2V_EINVAL, "corpus is NULL");
  if (c.table == nullptr) return fail(W2V_EINVAL, "neg_table is NULL");
  if (c.T <= 0) return fail(W2V_EINVAL, "T must be positive");
  if (c.L < 1 || c.L > W2V_MAX_SENTENCE)
    return failf(W2V_EINVAL, "sentence_len must be in [1, %d]", W2V_MAX_SENTENCE);
  if (c.pos_begin < 0 || c.pos_end > c.T || c.pos_begin > c.pos_end)
    return fail(W2V_EINVAL, "need 0 <= pos_begin <= pos_end <= T");
  if (c.pos_begin % c.L != 0)
    return fail(W2V_EINVAL, "pos_begin must start a sentence");
  if (c.pos_end != c.T && c.pos_end % c.L != 0)
    return fail(W2V_EINVAL, "pos_end must end a sentence or equal T");
  if (c.V <= 0) return fail(W2V_EINVAL, "V must be positive");
  if (c.window < 1 || c.window > W2V_MAX_WINDOW)
    return failf(W2V_EINVAL, "window must be in [1, %d]", W2V_MAX_WINDOW);
  if (c.K < 0 || c.K > W2V_MAX_NEGATIVE)
    return failf(W2V_EINVAL, "K must be in [0, %d]", W2V_MAX_NEGATIVE);
  if (c.table_size <= 0 || c.table_size >= (int64_t(1) << 32))
    return fail(W2V_EINVAL, "table_size must be in [1, 2^32)");
  if (c.n_epochs < 1 || c.epoch < 0 || c.epoch >= c.n_epochs)
    return fail(W2V_EINVAL, "need 0 <= epoch < n_epochs");
  return W2V_OK;
}

static int check_matrices(const float* M_in, const float* M_out, int32_t V,
                          int32_t D, int32_t ld) {
  if (M_in == nullptr || M_out == nullptr)
    return fail(W2V_EINVAL, "M_in and M_out must not be NULL");
  if (V <= 0) return fail(W2V_EINVAL, "V must be positive");
  if (D < 1 || D > W2V_MAX_DIM)
    return failf(W2V_EINVAL, "D must be in [1, %d]", W2V_MAX_DIM);
  if (ld < D) return fail(W2V_EINVAL, "ld must be >= D");
  return W2V_OK;
}

// Ids below this never take a pending input-row slot: their updates go to
// the matrix at the end of every minibatch. These are the rows other
// sentences write constantly (atomic and split rows); with their updates
// held back, concurrent sentences keep stepping from stale values and the
// held-back steps add up, which makes a small vocabulary diverge.
static int pending_from(int hot_rows, int split_rows) {
  return hot_rows > split_rows ? hot_rows : split_rows;
}

static int epoch_blocks_per_cu(int C, int nmax, int window, int K) {
  (void)window;
  return train_blocks_per_cu(C, nmax, K);
}

// Concurrency cap of a default launch (max_inflight = 0) for a vocabulary
// of V words: V / (4 G (2 window + K + 1)), at least 1. A minibatch holds
// up to 2 window input rows and K + 1 output rows while it computes; a
// group of G targets holds about G times as many and takes its step from
// rows G targets old. With the cap, the rows the concurrent sentences hold
// at once stay under a quarter of the vocabulary, so few of them are read
// stale. Measured on 200,000 tokens over 1,000 words (200 sentences, cap
// 15): the training loss of every tenth of the epoch within 0.4% of the
// sequential epoch, against up to 12% apart with all 200 sentences in
// flight. At 10^6 words the cap (15,625) is above what the GPU holds.
static int64_t vocab_inflight_cap(int64_t V, int window, int K, int group) {
  const int64_t per = 4 * (int64_t)group * (2 * (int64_t)window + K + 1);
  const int64_t cap = V / per;
  return cap > 0 ? cap : 1;
}

// Concurrency cap of a default launch for K negatives: 131072 / (K + 1)
// (2016 at K = 64; above what the GPU holds for K <= 40). Under a Zipf law
// the most frequent words are drawn as negatives by most minibatches once K
// is large, so the rows of those words take one update from nearly every
// sentence in flight, each computed from the row as it was before the
// others landed; past some number of such concurrent updates the Hogwild
// epoch overshoots and diverges. Measured on 1e8 tokens over 10^6 words
// (Zipf(1.07), window 5, alpha 0.025, the conflict model's atomic rows and
// split head): at D = 100, K = 64 finite and learning with 1024, 1536 and
// 2048 sentences in flight, NaN with 2560 and 3072; at D = 300, K = 64
// finite up to 3072; at K <= 15 finite at every concurrency the GPU holds.
// (At twice that learning rate, K = 15 diverged with 3072 in flight: the
// bound is the method's, and a caller who raises alpha or the concurrency
// checks the loss with w2v_check_loss.)
static int64_t negatives_inflight_cap(int K) {
  const int64_t cap = (int64_t)131072 / ((int64_t)K + 1);
  return cap > 0 ? cap : 1;
}

// A default launch also runs its sentences in at least kMinRounds rounds of
// the persistent grid, so that most sentences start from a model that the
// earlier ones have moved: with every sentence of a short range in flight at
// once, each starts from the initial model and the range behaves like one
// large stale batch (40 sentences over 3,000 words, all in flight: held-out
// loss 3% above the sequential epoch).
constexpr int64_t kMinRounds = 8;

static int64_t rounds_inflight_cap(int64_t n_sent) {
  const int64_t cap = (n_sent + kMinRounds - 1) / kMinRounds;
  return cap > 0 ? cap : 1;
}

}  // namespace w2v

using namespace w2v;

extern "C" {

int w2v_version(void) { return 104; }

const char* w2v_last_error(void) { return g_error; }

int w2v_init(void) {
  int dev = 0;
  int rc = current_device(dev);
  if (rc != W2V_OK) return rc;
  std::lock_guard<std::mutex> lock(g_dev_mu);
  rc = setup_device_locked(dev);
  return rc == W2V_OK ? ok() : rc;
}

int w2v_device_status(void* stream) {
  hipError_t e = hipStreamSynchronize((hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  int32_t* unused = nullptr;
  const int rc = enter_device(&unused);
  return rc == W2V_OK ? ok() : rc;
}

int w2v_check_loss(const double* loss_buckets, int32_t n_buckets, void* stream) {
  if (n_buckets < 0) return fail(W2V_EINVAL, "n_buckets must be >= 0");
  if (n_buckets > 0 && loss_buckets == nullptr)
    return fail(W2V_EINVAL, "loss_buckets is NULL");
  if (n_buckets == 0) return ok();
  const size_t bytes = sizeof(double) * 2 * (size_t)n_buckets;
  double* h = (double*)malloc(bytes);
  if (h == nullptr) return fail(W2V_ENOMEM, "host copy of the loss buckets");
  hipError_t e = hipMemcpyAsync(h, loss_buckets, bytes, hipMemcpyDeviceToHost,
                                (hipStream_t)stream);
  if (e == hipSuccess) e = hipStreamSynchronize((hipStream_t)stream);
  if (e != hipSuccess) {
    free(h);
    return hip_fail(e, "copy of the loss buckets");
  }
  for (int32_t b = 0; b < n_buckets; ++b) {
    const double sum = h[2 * b], cnt = h[2 * b + 1];
    if (!__builtin_isfinite(sum) || !__builtin_isfinite(cnt)) {
      free(h);
      return failf(W2V_ENONFINITE,
                   "loss bucket %d is not finite (sum %g over %g input words): a NaN "
                   "or Inf reached the rows its minibatches read",
                   (int)b, sum, cnt);
    }
  }
  free(h);
  return ok();
}

int w2v_build_tables(const int64_t* counts, int32_t V, double neg_power,
                     double sample_t, int32_t* neg_table, int64_t table_size,
                     uint32_t* keep_thresh) {
  return build_tables(counts, V, neg_power, sample_t, neg_table, table_size,
                      keep_thresh);
}

int32_t w2v_hot_rows(const int64_t* counts, int32_t V, double neg_power,
                     double sample_t, int32_t window, int32_t K,
                     int64_t inflight, double tol) {
  return hot_rows(counts, V, neg_power, sample_t, window, K, inflight, tol);
}

int64_t w2v_default_inflight(int32_t V, int32_t D, int32_t window, int32_t K,
                             int32_t group) {
  if (V <= 0) return fail(W2V_EINVAL, "V must be positive");
  if (group != 1 && group != 2 && group != 4 && group != 8)
    return fail(W2V_EINVAL, "group must be 1, 2, 4 or 8");
  if (D < 1 || D > W2V_MAX_DIM)
    return failf(W2V_EINVAL, "D must be in [1, %d]", W2V_MAX_DIM);
  if (window < 1 || window > W2V_MAX_WINDOW)
    return failf(W2V_EINVAL, "window must be in [1, %d]", W2V_MAX_WINDOW);
  if (K < 0 || K > W2V_MAX_NEGATIVE)
    return failf(W2V_EINVAL, "K must be in [0, %d]", W2V_MAX_NEGATIVE);
  const int C = columns_for(D);
  const int nmax = inputs_cap_for(2 * window);
  if (C == 0 || nmax == 0 || !train_shape_supported(C, nmax))
    return failf(W2V_EUNSUPPORTED, "no compiled kernel for D=%d window=%d", D,
                 window);
  const int omax = group > 1 ? group_outputs_cap_for(group + K) : 0;
  const int per_cu = group > 1 ? grouped_blocks_per_cu(C, omax, K)
                               : epoch_blocks_per_cu(C, nmax, window, K);
  const int cus = cu_count();
  if (per_cu <= 0 || cus <= 0) return fail(W2V_EHIP, "device query failed");
  ok();
  const int64_t full = (int64_t)per_cu * cus;
  int64_t cap = vocab_inflight_cap(V, window, K, group);
  const int64_t ncap = negatives_inflight_cap(K);
  if (ncap < cap) cap = ncap;
  return full < cap ? full : cap;
}

int32_t w2v_pending_slots(int32_t D, int32_t window, int32_t K) {
  if (D < 1 || D > W2V_MAX_DIM)
    return failf(W2V_EINVAL, "D must be in [1, %d]", W2V_MAX_DIM);
  if (window < 1 || window > W2V_MAX_WINDOW)
    return failf(W2V_EINVAL, "window must be in [1, %d]", W2V_MAX_WINDOW);
  if (K < 0 || K > W2V_MAX_NEGATIVE)
    return failf(W2V_EINVAL, "K must be in [0, %d]", W2V_MAX_NEGATIVE);
  const int C = columns_for(D);
  const int nmax = inputs_cap_for(2 * window);
  if (C == 0 || nmax == 0 || !train_shape_supported(C, nmax))
    return failf(W2V_EUNSUPPORTED, "no compiled kernel for D=%d window=%d", D,
                 window);
  ok();
  return train_pending_slots(C, nmax, K);
}

}  // extern "C"

namespace w2v {

// w2v_train_epoch and w2v_train_epoch_noalloc: with `noalloc` the partial
// rows live in the device's scratch array instead of the caller's workspace.
static int train_epoch_impl(const int32_t* corpus, int64_t T, int64_t pos_begin,
                            int64_t pos_end, int32_t sentence_len, float* M_in,
                            float* M_out, int32_t V, int32_t D, int32_t ld,
                            int32_t window, int32_t K, const int32_t* neg_table,
                            int64_t table_size, const uint32_t* keep_thresh,
                            float alpha0, float min_alpha_frac, int32_t epoch,
                            int32_t n_epochs, uint64_t seed, double* loss_buckets,
                            int32_t n_buckets, int64_t* stats, int32_t max_inflight,
                            int32_t hot_rows, int32_t split_rows, void* workspace,
                            size_t workspace_bytes, int32_t algorithm, int32_t group,
                            void* stream, bool noalloc) {
  int rc = check_sampling({corpus, T, pos_begin, pos_end, sentence_len, V,
                           window, K, neg_table, table_size, epoch, n_epochs});
  if (rc != W2V_OK) return rc;
  rc = check_matrices(M_in, M_out, V, D, ld);
  if (rc != W2V_OK) return rc;
  if (loss_buckets != nullptr && n_buckets < 1)
    return fail(W2V_EINVAL, "n_buckets must be >= 1 with loss_buckets");
  if (max_inflight < 0) return fail(W2V_EINVAL, "max_inflight must be >= 0");
  if (hot_rows < 0) return fail(W2V_EINVAL, "hot_rows must be >= 0");
  if (algorithm != W2V_ALGORITHM_HOGBATCH && algorithm != W2V_ALGORITHM_PAIRWISE &&
      algorithm != W2V_ALGORITHM_HOGBATCH_IMMEDIATE)
    return fail(W2V_EINVAL,
                "algorithm must be W2V_ALGORITHM_HOGBATCH, _PAIRWISE or _HOGBATCH_IMMEDIATE");
  if (split_rows < 0 || split_rows > V)
    return fail(W2V_EINVAL, "split_rows must be in [0, V]");
  if (algorithm == W2V_ALGORITHM_PAIRWISE && split_rows != 0)
    return fail(W2V_EINVAL, "split_rows must be 0 with the pairwise algorithm");
  if (group != 1 && group != 2 && group != 4 && group != 8)
    return fail(W2V_EINVAL, "group must be 1, 2, 4 or 8");
  if (group > 1 && algorithm == W2V_ALGORITHM_PAIRWISE)
    return fail(W2V_EINVAL, "group > 1 needs the HogBatch algorithm");
  if (group > 1 && (group * 2 * window > 64 || 2 * window + group > 32 ||
                    group + K > 32))
    return fail(W2V_EINVAL,
                "group needs 2 window group <= 64, 2 window + group <= 32 and "
                "group + K <= 32");
  if (noalloc && w2v_train_epoch_workspace_bytes(split_rows, ld) > W2V_NOALLOC_SCRATCH_BYTES)
    return failf(W2V_EINVAL,
                 "split_rows = %d at ld = %d needs %zu bytes of partial rows, more than "
                 "the %d bytes of scratch of w2v_train_epoch_noalloc",
                 split_rows, ld, w2v_train_epoch_workspace_bytes(split_rows, ld),
                 W2V_NOALLOC_SCRATCH_BYTES);
  if (split_rows > 0 && !noalloc) {
    if (workspace == nullptr) return fail(W2V_EINVAL, "workspace is NULL");
    if (workspace_bytes < w2v_train_epoch_workspace_bytes(split_rows, ld))
      return fail(W2V_EINVAL, "workspace too small for split_rows");
    if (((uintptr_t)workspace & 255u) != 0)
      return fail(W2V_EINVAL, "workspace must be 256-byte aligned");
  }
  const bool pairwise = algorithm == W2V_ALGORITHM_PAIRWISE;
  const bool grouped = group > 1;
  const int C = columns_for(D);
  const int nmax = inputs_cap_for(2 * window);
  // a group's output columns: its targets and the shared negatives
  const int omax = grouped ? group_outputs_cap_for(group + K) : 0;
  // Algorithm 1 handles one input word at a time and a group its input rows
  // in blocks: D (and a group's output columns) limit them.
  const bool shape_ok = pairwise  ? C != 0
                        : grouped ? C != 0 && grouped_shape_supported(C, omax)
                                  : C != 0 && nmax != 0 && train_shape_supported(C, nmax);
  if (!shape_ok)
    return failf(W2V_EUNSUPPORTED, "no compiled kernel for D=%d window=%d", D,
                 window);
  int32_t* status = nullptr;
  void* scratch_dev = nullptr;
  rc = enter_device(&status, &scratch_dev, noalloc);
  if (rc != W2V_OK) return rc;
  if (noalloc) workspace = scratch_dev;
  const int64_t n_sent = (pos_end - pos_begin + sentence_len - 1) / sentence_len;
  if (n_sent == 0) return ok();

  EpochArgs a{};
  a.corpus = corpus;
  a.T = T;
  a.pos_begin = pos_begin;
  a.pos_end = pos_end;
  a.n_sent = n_sent;
  a.L = sentence_len;
  a.status = status;
  a.M_in = M_in;
  a.M_out = M_out;
  a.V = V;
  a.D = D;
  a.ld = ld;
  a.w = window;
  a.K = K;
  a.table = neg_table;
  a.table_size = table_size;
  a.thr = keep_thresh;
  a.alpha0 = alpha0;
  a.min_frac = min_alpha_frac;
  a.epoch = epoch;
  a.n_epochs = n_epochs;
  a.seed = seed;
  a.loss = loss_buckets;
  a.n_buckets = n_buckets;
  a.stats = stats;
  a.hot_rows = hot_rows;
  a.split_rows = split_rows;
  a.part = (float*)workspace;
  a.group = group;
  a.pend_slots = (pairwise || grouped || algorithm == W2V_ALGORITHM_HOGBATCH_IMMEDIATE)
                     ? 0
                     : train_pending_slots(C, nmax, K);
  a.pend_from = pending_from(hot_rows, split_rows);
  a.target_batch = (pairwise || grouped) ? 64 : train_target_batch(C, nmax, K);

  int64_t grid = max_inflight;
  if (grid == 0) {
    const int per_cu = pairwise  ? pairwise_blocks_per_cu(C, K)
                       : grouped ? grouped_blocks_per_cu(C, omax, K)
                                 : epoch_blocks_per_cu(C, nmax, window, K);
    const int cus = cu_count();
    grid = (int64_t)(per_cu > 0 ? per_cu : 1) * (cus > 0 ? cus : 1);
    const int64_t cap = vocab_inflight_cap(V, window, K, group);
    if (grid > cap) grid = cap;
    const int64_t ncap = negatives_inflight_cap(K);
    if (grid > ncap) grid = ncap;
    const int64_t rcap = rounds_inflight_cap(n_sent);
    if (grid > rcap) grid = rcap;
  }
  if (grid > n_sent) grid = n_sent;
  if (grid > (1 << 30)) grid = 1 << 30;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = hipSuccess;
  if (split_rows > 0) {
    e = launch_part_clear(a, s);
    if (e != hipSuccess) return hip_fail(e, "partial-row clear launch");
  }
  e = pairwise  ? launch_pairwise(C, a, (int)grid, s)
      : grouped ? launch_grouped(C, omax, a, (int)grid, s)
                : launch_train(C, nmax, a, (int)grid, s);
  if (e != hipSuccess) return hip_fail(e, "train kernel launch");
  if (split_rows > 0) {
    e = launch_part_fold(a, s);
    if (e != hipSuccess) return hip_fail(e, "partial-row fold launch");
  }
  return ok();
}

}  // namespace w2v

extern "C" {

int w2v_train_epoch(const int32_t* corpus, int64_t T, int64_t pos_begin,
                    int64_t pos_end, int32_t sentence_len, float* M_in,
                    float* M_out, int32_t V, int32_t D, int32_t ld,
                    int32_t window, int32_t K, const int32_t* neg_table,
                    int64_t table_size, const uint32_t* keep_thresh,
                    float alpha0, float min_alpha_frac, int32_t epoch,
                    int32_t n_epochs, uint64_t seed, double* loss_buckets,
                    int32_t n_buckets, int64_t* stats, int32_t max_inflight,
                    int32_t hot_rows, int32_t split_rows, void* workspace,
                    size_t workspace_bytes, int32_t algorithm, int32_t group,
                    void* stream) {
  return train_epoch_impl(corpus, T, pos_begin, pos_end, sentence_len, M_in, M_out, V,
                          D, ld, window, K, neg_table, table_size, keep_thresh, alpha0,
                          min_alpha_frac, epoch, n_epochs, seed, loss_buckets, n_buckets,
                          stats, max_inflight, hot_rows, split_rows, workspace,
                          workspace_bytes, algorithm, group, stream, false);
}

int w2v_train_epoch_noalloc(const int32_t* corpus, int64_t T, int64_t pos_begin,
                            int64_t pos_end, int32_t sentence_len, float* M_in,
                            float* M_out, int32_t V, int32_t D, int32_t ld,
                            int32_t window, int32_t K, const int32_t* neg_table,
                            int64_t table_size, const uint32_t* keep_thresh,
                            float alpha0, float min_alpha_frac, int32_t epoch,
                            int32_t n_epochs, uint64_t seed, double* loss_buckets,
                            int32_t n_buckets, int64_t* stats, int32_t max_inflight,
                            int32_t hot_rows, int32_t split_rows, int32_t algorithm,
                            int32_t group, void* stream) {
  return train_epoch_impl(corpus, T, pos_begin, pos_end, sentence_len, M_in, M_out, V,
                          D, ld, window, K, neg_table, table_size, keep_thresh, alpha0,
                          min_alpha_frac, epoch, n_epochs, seed, loss_buckets, n_buckets,
                          stats, max_inflight, hot_rows, split_rows, nullptr, 0,
                          algorithm, group, stream, true);
}

size_t w2v_train_epoch_workspace_bytes(int32_t split_rows, int32_t ld) {
  if (split_rows <= 0 || ld <= 0) return 0;
  return (size_t)2 * (size_t)split_rows * W2V_SPLIT_PARTS * (size_t)ld *
         sizeof(float);
}

int w2v_debug_minibatches(const int32_t* corpus, int64_t T, int64_t pos_begin,
                          int64_t pos_end, int32_t sentence_len, int32_t V,
                          int32_t window, int32_t K, const int32_t* neg_table,
                          int64_t table_size, const uint32_t* keep_thresh,
                          float alpha0, float min_alpha_frac, int32_t epoch,
                          int32_t n_epochs, uint64_t seed, int32_t* out_targets,
                          int32_t* out_ctx, int32_t* out_negs,
                          uint8_t* out_mask, float* out_alpha, int64_t* stats,
                          void* stream) {
  int rc = check_sampling({corpus, T, pos_begin, pos_end, sentence_len, V,
                           window, K, neg_table, table_size, epoch, n_epochs});
  if (rc != W2V_OK) return rc;
  if (out_targets == nullptr || out_ctx == nullptr || out_alpha == nullptr ||
      (K > 0 && (out_negs == nullptr || out_mask == nullptr)))
    return fail(W2V_EINVAL, "output pointers must not be NULL");
  int32_t* status = nullptr;
  rc = enter_device(&status);
  if (rc != W2V_OK) return rc;
  const int64_t n_sent = (pos_end - pos_begin + sentence_len - 1) / sentence_len;
  if (n_sent == 0) return ok();
  EpochArgs a{};
  a.status = status;
  a.corpus = corpus;
  a.T = T;
  a.pos_begin = pos_begin;
  a.pos_end = pos_end;
  a.n_sent = n_sent;
  a.L = sentence_len;
  a.V = V;
  a.D = 1;
  a.ld = 1;
  a.w = window;
  a.K = K;
  a.table = neg_table;
  a.table_size = table_size;
  a.thr = keep_thresh;
  a.alpha0 = alpha0;
  a.min_frac = min_alpha_frac;
  a.epoch = epoch;
  a.n_epochs = n_epochs;
  a.seed = seed;
  a.stats = stats;
  a.out_targets = out_targets;
  a.out_ctx = out_ctx;
  a.out_negs = out_negs;
  a.out_mask = out_mask;
  a.out_alpha = out_alpha;
  int64_t grid = n_sent < (1 << 20) ? n_sent : (1 << 20);
  hipError_t e = launch_export(a, (int)grid, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "export kernel launch");
  return ok();
}

size_t w2v_step_batch_workspace_bytes(int32_t V, int32_t ld) {
  if (V <= 0 || ld <= 0) return 0;
  const size_t one = (size_t)V * (size_t)ld * sizeof(double);
  const size_t aligned = (one + 255) / 256 * 256;
  return 2 * aligned;
}

int w2v_step_batch(int32_t B, int32_t N, int32_t K, const int32_t* targets,
                   const int32_t* contexts, const int32_t* negatives,
                   const float* alpha, float alpha_scalar, float* M_in,
                   float* M_out, int32_t V, int32_t D, int32_t ld,
                   void* workspace, size_t workspace_bytes, int64_t* stats,
                   void* stream) {
  if (B < 0) return fail(W2V_EINVAL, "B must be >= 0");
  if (N < 0 || N > W2V_MAX_BATCH_INPUTS)
    return failf(W2V_EINVAL, "N must be in [0, %d]", W2V_MAX_BATCH_INPUTS);
  if (K < 0 || K > W2V_MAX_NEGATIVE)
    return failf(W2V_EINVAL, "K must be in [0, %d]", W2V_MAX_NEGATIVE);
  int rc = check_matrices(M_in, M_out, V, D, ld);
  if (rc != W2V_OK) return rc;
  if (B > 0 && targets == nullptr) return fail(W2V_EINVAL, "targets is NULL");
  if (B > 0 && N > 0 && contexts == nullptr)
    return fail(W2V_EINVAL, "contexts is NULL");
  if (B > 0 && K > 0 && negatives == nullptr)
    return fail(W2V_EINVAL, "negatives is NULL");
  const size_t need = w2v_step_batch_workspace_bytes(V, ld);
  if (workspace == nullptr || workspace_bytes < need)
    return failf(W2V_EINVAL, "workspace must hold %zu bytes", need);
  if (((uintptr_t)workspace & 255u) != 0)
    return fail(W2V_EINVAL, "workspace must be 256-byte aligned");
  const int C = columns_for(D);
  const int nmax = inputs_cap_for(N > 0 ? N : 1);
  if (C == 0 || nmax == 0 || !train_shape_supported(C, nmax))
    return failf(W2V_EUNSUPPORTED, "no compiled kernel for D=%d N=%d", D, N);
  int32_t* status = nullptr;
  rc = enter_device(&status);
  if (rc != W2V_OK) return rc;
  if (B == 0 || N == 0) return ok();

  hipStream_t s = (hipStream_t)stream;

  StepArgs a{};
  a.status = status;
  a.B = B;
  a.N = N;
  a.K = K;
  a.targets = targets;
  a.contexts = contexts;
  a.negatives = negatives;
  a.alpha = alpha;
  a.alpha_scalar = alpha_scalar;
  a.M_in = M_in;
  a.dM_in = (double*)workspace;
  a.dM_out = (double*)((char*)workspace + need / 2);
  a.M_out = M_out;
  a.V = V;
  a.D = D;
  a.ld = ld;
  a.stats = stats;
  const int grid = B < (1 << 20) ? B : (1 << 20);
  hipError_t e = launch_step(C, nmax, a, grid, s);
  if (e != hipSuccess) return hip_fail(e, "step kernel launch");
  return ok();
}

size_t w2v_step_batch_sorted_workspace_bytes(int32_t B, int32_t N, int32_t K,
                                             int32_t V, int32_t ld) {
  if (B < 0 || N < 0 || K < 0 || V <= 0 || ld <= 0) return 0;
  return sorted_step_workspace_bytes(B, N, K, V, ld);
}

int w2v_step_batch_sorted(int32_t B, int32_t N, int32_t K, const int32_t* targets,
                          const int32_t* contexts, const int32_t* negatives,
                          const float* alpha, float alpha_scalar, float* M_in,
                          float* M_out, int32_t V, int32_t D, int32_t ld,
                          void* workspace, size_t workspace_bytes, int64_t* stats,
                          void* stream) {
  if (B < 0) return fail(W2V_EINVAL, "B must be >= 0");
  if (N < 0 || N > W2V_MAX_BATCH_INPUTS)
    return failf(W2V_EINVAL, "N must be in [0, %d]", W2V_MAX_BATCH_INPUTS);
  if (K < 0 || K > W2V_MAX_NEGATIVE)
    return failf(W2V_EINVAL, "K must be in [0, %d]", W2V_MAX_NEGATIVE);
  if ((int64_t)B * (N + K + 1) > INT32_MAX)
    return fail(W2V_EINVAL, "B * (N + K + 1) must fit in int32");
  int rc = check_matrices(M_in, M_out, V, D, ld);
  if (rc != W2V_OK) return rc;
  if (B > 0 && targets == nullptr) return fail(W2V_EINVAL, "targets is NULL");
  if (B > 0 && N > 0 && contexts == nullptr)
    return fail(W2V_EINVAL, "contexts is NULL");
  if (B > 0 && K > 0 && negatives == nullptr)
    return fail(W2V_EINVAL, "negatives is NULL");
  const size_t need = w2v_step_batch_sorted_workspace_bytes(B, N, K, V, ld);
  if (need == 0) return fail(W2V_EHIP, "sort size query failed");
  if (workspace == nullptr || workspace_bytes < need)
    return failf(W2V_EINVAL, "workspace must hold %zu bytes", need);
  if (((uintptr_t)workspace & 255u) != 0)
    return fail(W2V_EINVAL, "workspace must be 256-byte aligned");
  const int C = columns_for(D);
  const int nmax = inputs_cap_for(N > 0 ? N : 1);
  if (C == 0 || nmax == 0 || !sorted_step_supported(C, nmax))
    return failf(W2V_EUNSUPPORTED, "no compiled kernel for D=%d N=%d", D, N);
  int32_t* status = nullptr;
  rc = enter_device(&status);
  if (rc != W2V_OK) return rc;
  if (B == 0 || N == 0) return ok();

  SortedStepArgs a{};
  a.status = status;
  a.B = B;
  a.N = N;
  a.K = K;
  a.targets = targets;
  a.contexts = contexts;
  a.negatives = negatives;
  a.alpha = alpha;
  a.alpha_scalar = alpha_scalar;
  a.M_in = M_in;
  a.M_out = M_out;
  a.V = V;
  a.D = D;
  a.ld = ld;
  a.stats = stats;
  hipError_t e = launch_step_sorted(C, nmax, a, workspace, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "sorted step launch");
  return ok();
}

size_t w2v_build_vocab_workspace_bytes(int32_t V_raw, int64_t T) {
  if (V_raw <= 0 || T < 0) return 0;
  return vocab_workspace_bytes(V_raw, T);
}

int w2v_build_vocab(const int32_t* raw, int64_t T, int32_t V_raw,
                    int64_t min_count, int64_t* ranked_counts,
                    int32_t* rank_of, int32_t* v_kept, int32_t* corpus_out,
                    void* workspace, size_t workspace_bytes, void* stream) {
  if (T < 0) return fail(W2V_EINVAL, "T must be >= 0");
  if (T > 0 && raw == nullptr) return fail(W2V_EINVAL, "raw is NULL");
  if (V_raw <= 0) return fail(W2V_EINVAL, "V_raw must be positive");
  if (min_count < 0) return fail(W2V_EINVAL, "min_count must be >= 0");
  if (ranked_counts == nullptr || rank_of == nullptr || v_kept == nullptr)
    return fail(W2V_EINVAL, "ranked_counts, rank_of and v_kept must not be NULL");
  if (workspace == nullptr || workspace_bytes < w2v_build_vocab_workspace_bytes(V_raw, T))
    return failf(W2V_EINVAL, "workspace must hold %zu bytes",
                 w2v_build_vocab_workspace_bytes(V_raw, T));
  if (((uintptr_t)workspace & 255u) != 0)
    return fail(W2V_EINVAL, "workspace must be 256-byte aligned");
  int32_t* status = nullptr;
  const int rc = enter_device(&status);
  if (rc != W2V_OK) return rc;
  hipError_t e = launch_vocab(raw, T, V_raw, min_count, ranked_counts, rank_of,
                              v_kept, corpus_out, workspace, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "vocabulary launch");
  return ok();
}

}  // extern "C"
