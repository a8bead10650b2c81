// C ABI of the Fork-dLLM step (declared in include/fork_step.h): argument
// validation, the library-managed workspace, and the three launches
//   gemm_stats (LM head + per-tile statistics) -> merge -> select
// enqueued on the caller's stream.
#include "fork_step.h"

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>

#include <mutex>
#include <vector>

#include "fork_kernels.h"
#include "workspace_registry.h"

// Device scratch of fork_step_noalloc: a static array that every GPU the
// library runs on holds (its own copy) until the process ends.  Host code
// never uses the array's name as a device address: the address of each
// device's copy comes from hipGetSymbolAddress (scratch_address below).
static __device__ __align__(256) unsigned char scratch[FORK_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kVersion = 1 * 10000 + 1 * 100 + 0;
constexpr size_t kAlign = 256;
// Per-tile byte offsets of the LM-head kernel are 32-bit: 256 rows x d x 4 B
// must stay below 2^31.
constexpr int kMaxD = 1 << 20;

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Workspace layout: [partials: nvt*M float4][argmax: M int32]
// [rows: M int32 (active-row list or row map)][drawn partials: nvt*M float4,
// only when candidates are drawn].
struct Layout {
  size_t partial_off, argmax_off, rows_off, spartial_off, total;
};

bool layout_for(int32_t B, int32_t L, int32_t V, bool sampling, Layout* out) {
  if (B <= 0 || L <= 0 || V <= 0) return false;
  const long long M = (long long)B * L;
  if (M > 0x7fffffffLL) return false;
  const size_t nvt = (size_t)fork::num_vocab_tiles(V);
  const size_t part = align_up(nvt * (size_t)M * sizeof(float4));
  out->partial_off = 0;
  out->argmax_off = part;
  out->rows_off = out->argmax_off + align_up((size_t)M * sizeof(int32_t));
  out->spartial_off = out->rows_off + align_up((size_t)M * sizeof(int32_t));
  out->total = out->spartial_off + (sampling ? part : 0);
  return true;
}

// hipMalloc / hipFree / hipDeviceSynchronize on a given device, restoring
// the caller's current device.
struct HipBackend {
  static int alloc(int dev, size_t bytes, void** out) {
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) return FORK_EHIP;
    if (cur != dev && hipSetDevice(dev) != hipSuccess) return FORK_EHIP;
    const hipError_t e = hipMalloc(out, bytes);
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || !*out) {
      fail(FORK_ENOMEM, "hipMalloc(%zu) for the workspace: %s", bytes, hipGetErrorString(e));
      return FORK_ENOMEM;
    }
    return 0;
  }
  static void free(int dev, void* p) {
    int cur = 0;
    const bool have = hipGetDevice(&cur) == hipSuccess;
    if (hipSetDevice(dev) == hipSuccess) (void)hipFree(p);
    if (have) (void)hipSetDevice(cur);
  }
  static void sync(int dev) {
    int cur = 0;
    const bool have = hipGetDevice(&cur) == hipSuccess;
    if (hipSetDevice(dev) == hipSuccess) (void)hipDeviceSynchronize();
    if (have) (void)hipSetDevice(cur);
  }
};

fork::WorkspaceRegistry<HipBackend> g_registry;

// The device a stream belongs to (the current device for the NULL stream).
int stream_device(hipStream_t stream, int* dev) {
  hipError_t e = stream ? hipStreamGetDevice(stream, dev) : hipGetDevice(dev);
  if (e != hipSuccess) return fail(FORK_EHIP, "device of the stream: %s", hipGetErrorString(e));
  return FORK_OK;
}

// The library-managed buffer of (device of `stream`, `stream`), grown to
// `need` bytes, with *lock holding the registry until the caller's launches
// are enqueued.  Refused while the stream is being captured into a graph: a
// graph would keep the buffer's address past fork_release.
int get_workspace(hipStream_t stream, size_t need, void** out, std::unique_lock<std::mutex>* lock) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  hipError_t e = hipStreamIsCapturing(stream, &cs);
  if (e != hipSuccess) return fail(FORK_EHIP, "hipStreamIsCapturing: %s", hipGetErrorString(e));
  if (cs != hipStreamCaptureStatusNone)
    return fail(FORK_EINVAL,
                "the stream is being captured into a graph: pass a caller workspace "
                "(workspace / workspace_bytes) that outlives the graph");
  int dev = 0;
  int rc = stream_device(stream, &dev);
  if (rc != FORK_OK) return rc;
  rc = g_registry.acquire(dev, reinterpret_cast<uintptr_t>(stream), need, out, lock);
  if (rc != 0) return rc == FORK_ENOMEM ? FORK_ENOMEM : fail(FORK_EHIP, "workspace allocation failed");
  return FORK_OK;
}

constexpr int kMaxDevices = 256;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};  // device address of `scratch`, per device

// Address of device `dev`'s copy of `scratch`, looked up once per device
// (with that device current) and kept.
int scratch_address(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return fail(FORK_EINVAL, "device %d out of range", dev);
  std::lock_guard<std::mutex> g(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    int cur = 0;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return fail(FORK_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess)
      return fail(FORK_EHIP, "hipSetDevice(%d): %s", dev, hipGetErrorString(e));
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || !p)
      return fail(FORK_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                  hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return FORK_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Smallest positive sampling temperature: below it 1/tau overflows the
// Gumbel keys.
constexpr float kMinTemperature = 1e-30f;

// The LM-head launch has one 512-thread workgroup per (vocabulary tile,
// position tile); its work-item count must stay below 2^32.
bool grid_fits(long long positions, int V) {
  const long long tiles = (long long)fork::num_vocab_tiles(V) * ((positions + fork::kTileP - 1) / fork::kTileP);
  return tiles * 512 < (1LL << 32);
}

int validate(const fork_step_args* a) {
  if (!a) return fail(FORK_EINVAL, "args is NULL");
  if (a->B < 0 || a->L <= 0 || a->d <= 0 || a->V <= 0)
    return fail(FORK_EINVAL, "need B >= 0 and L, d, V > 0 (B=%d L=%d d=%d V=%d)", a->B, a->L,
                a->d, a->V);
  if (a->B > 0 && (!a->hidden || !a->W_head || !a->tokens || !a->mask || !a->block_start ||
                   !a->out_conf || !a->out_entropy || !a->out_logp || !a->out_fallback))
    return fail(FORK_EINVAL, "a required pointer is NULL");
  if ((long long)a->B * a->L > 0x7fffffffLL)
    return fail(FORK_EINVAL, "B*L = %lld does not fit int32", (long long)a->B * a->L);
  if (a->block_len <= 0 || a->block_len > a->L)
    return fail(FORK_EINVAL, "block_len=%d must lie in [1, L=%d]", a->block_len, a->L);
  if (!isfinite(a->tau)) return fail(FORK_EINVAL, "tau must be finite");
  if (a->dtype != FORK_BF16 && a->dtype != FORK_F32)
    return fail(FORK_EINVAL, "unknown dtype %d", a->dtype);
  if (a->rule < FORK_RULE_LEFTMOST || a->rule > FORK_RULE_RANDOM)
    return fail(FORK_EINVAL, "unknown fallback rule %d", a->rule);
  if (a->rule == FORK_RULE_RANDOM && a->B > 0 && !a->fallback_uniform)
    return fail(FORK_EINVAL, "FORK_RULE_RANDOM needs fallback_uniform");
  if (a->dtype == FORK_BF16 && a->d % 8 != 0)
    return fail(FORK_EUNSUPPORTED, "bf16 path needs d %% 8 == 0 (d=%d)", a->d);
  if (a->dtype == FORK_F32 && a->d % 4 != 0)
    return fail(FORK_EUNSUPPORTED, "fp32 path needs d %% 4 == 0 (d=%d)", a->d);
  if (a->d > kMaxD)
    return fail(FORK_EUNSUPPORTED, "d=%d exceeds the supported maximum %d", a->d, kMaxD);
  if (!aligned16(a->hidden) || !aligned16(a->W_head))
    return fail(FORK_EINVAL, "hidden and W_head must be 16-byte aligned");
  if (a->rows_mode != FORK_ROWS_ALL && a->rows_mode != FORK_ROWS_ACTIVE)
    return fail(FORK_EINVAL, "unknown rows_mode %d", a->rows_mode);
  if (a->rows_mode == FORK_ROWS_ACTIVE &&
      (long long)a->B * a->L * a->d * (a->dtype == FORK_BF16 ? 2 : 4) >= (1LL << 31))
    return fail(FORK_EUNSUPPORTED, "FORK_ROWS_ACTIVE needs B*L*d*element_size < 2^31");
  if (!(a->sample_temperature >= 0.0f) || !isfinite(a->sample_temperature))
    return fail(FORK_EINVAL, "sample_temperature must be finite and >= 0");
  if (a->sample_temperature > 0.0f && a->sample_temperature < kMinTemperature)
    return fail(FORK_EINVAL, "sample_temperature must be 0 or at least %g", (double)kMinTemperature);
  const int positions = a->rows_mode == FORK_ROWS_ACTIVE ? a->B * a->block_len : a->B * a->L;
  if (!grid_fits(positions, a->V))
    return fail(FORK_EUNSUPPORTED, "%d positions x V=%d exceed one launch grid; split the batch",
                positions, a->V);
  return FORK_OK;
}

// The launches of one step (active rows, LM head, merge, selection) on
// the workspace `ws` laid out as `lay`; arguments already validated.
int enqueue_step(const fork_step_args* a, void* ws, const Layout& lay) {
  const bool sampling = a->sample_temperature > 0.0f;
  const int Mh = a->B * a->L;                       // rows of hidden
  const bool active = a->rows_mode == FORK_ROWS_ACTIVE;
  const int M = active ? a->B * a->block_len : Mh;  // positions through the LM head
  const int nvt = fork::num_vocab_tiles(a->V);
  float4* partials = reinterpret_cast<float4*>(static_cast<char*>(ws) + lay.partial_off);
  int32_t* argmax = a->out_argmax ? a->out_argmax
                                  : reinterpret_cast<int32_t*>(static_cast<char*>(ws) + lay.argmax_off);
  // one int32 region: the active-row list (FORK_ROWS_ACTIVE) or, when
  // drawing over all rows, the map of rows whose candidates are drawn
  int32_t* rows = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + lay.rows_off);
  int32_t* rowlist = active ? rows : nullptr;
  int32_t* rowmap = (!active && sampling) ? rows : nullptr;
  fork::SampleArgs sa = {};
  if (sampling) {
    sa.row = active ? rowlist : rowmap;
    sa.partials = reinterpret_cast<float4*>(static_cast<char*>(ws) + lay.spartial_off);
    sa.inv_tau = 1.0f / a->sample_temperature;
    sa.key0 = (uint32_t)a->sample_seed;
    sa.key1 = (uint32_t)(a->sample_seed >> 32);
    sa.counter = a->sample_counter;
  }
  hipStream_t stream = static_cast<hipStream_t>(a->stream);

  hipError_t e;
  if (rowlist || rowmap) {
    e = fork::launch_active_rows(a->B, a->L, a->block_len, a->mask, a->block_start, rowlist,
                                 rowmap, stream);
    if (e != hipSuccess) return fail(FORK_EHIP, "active_rows launch: %s", hipGetErrorString(e));
  }
  if (a->ev_lmhead_begin) {
    e = hipEventRecord(static_cast<hipEvent_t>(a->ev_lmhead_begin), stream);
    if (e != hipSuccess) return fail(FORK_EHIP, "hipEventRecord: %s", hipGetErrorString(e));
  }
  e = fork::launch_gemm_stats(a->hidden, a->W_head, a->dtype == FORK_BF16, M, a->d, a->V,
                              partials, rowlist, Mh, sa, fork::TargetArgs{}, stream);
  if (e != hipSuccess) return fail(FORK_EHIP, "gemm_stats launch: %s", hipGetErrorString(e));
  if (a->ev_lmhead_end) {
    e = hipEventRecord(static_cast<hipEvent_t>(a->ev_lmhead_end), stream);
    if (e != hipSuccess) return fail(FORK_EHIP, "hipEventRecord: %s", hipGetErrorString(e));
  }
  e = fork::launch_merge(partials, M, nvt, a->out_conf, a->out_entropy, a->out_logp, a->out_lse,
                         argmax, rowlist, sa.row, sa.partials, nullptr, nullptr, a->V, stream);
  if (e != hipSuccess) return fail(FORK_EHIP, "merge launch: %s", hipGetErrorString(e));
  e = fork::launch_select(a->B, a->L, a->block_len, a->tau, a->rule, a->out_conf,
                          a->out_entropy, a->fallback_uniform, argmax, a->tokens, a->mask,
                          a->block_start, a->out_fallback, a->out_ncommit, a->out_commit_pos,
                          /*position_major=*/false, stream);
  if (e != hipSuccess) return fail(FORK_EHIP, "select launch: %s", hipGetErrorString(e));

  static const bool sync_each = [] {
    const char* s = getenv("FORK_SYNC");
    return s && s[0] == '1';
  }();
  if (sync_each) {
    e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return fail(FORK_EHIP, "step failed: %s", hipGetErrorString(e));
  }
  return FORK_OK;
}

}  // namespace

extern "C" {

int fork_step_ex(const fork_step_args* a) {
  int rc = validate(a);
  if (rc != FORK_OK) return rc;
  if (a->B == 0) return FORK_OK;  // an empty batch: nothing to enqueue
  const bool sampling = a->sample_temperature > 0.0f;
  Layout lay;
  if (!layout_for(a->B, a->L, a->V, sampling, &lay)) return fail(FORK_EINVAL, "invalid sizes");
  void* ws = a->workspace;
  std::unique_lock<std::mutex> ws_lock;  // held until the launches are enqueued
  if (ws) {
    if (a->workspace_bytes < lay.total)
      return fail(FORK_EINVAL, "workspace holds %zu bytes, %zu needed", a->workspace_bytes, lay.total);
    if (((uintptr_t)ws % kAlign) != 0) return fail(FORK_EINVAL, "workspace must be 256-byte aligned");
  } else {
    rc = get_workspace(static_cast<hipStream_t>(a->stream), lay.total, &ws, &ws_lock);
    if (rc != FORK_OK) return rc;
  }
  return enqueue_step(a, ws, lay);
}

int fork_step_noalloc(const fork_step_args* a) {
  int rc = validate(a);
  if (rc != FORK_OK) return rc;
  if (a->workspace || a->workspace_bytes)
    return fail(FORK_EINVAL, "fork_step_noalloc uses the library's static scratch: "
                             "workspace must be NULL and workspace_bytes 0");
  if (a->B == 0) return FORK_OK;  // an empty batch: nothing to enqueue
  Layout lay;
  if (!layout_for(a->B, a->L, a->V, a->sample_temperature > 0.0f, &lay))
    return fail(FORK_EINVAL, "invalid sizes");
  if (lay.total > (size_t)FORK_NOALLOC_SCRATCH_BYTES)
    return fail(FORK_EUNSUPPORTED,
                "fork_step_noalloc: these sizes need %zu bytes of scratch, more than its "
                "maximum of %zu; use fork_step_ex with a workspace",
                lay.total, (size_t)FORK_NOALLOC_SCRATCH_BYTES);
  int dev = 0;
  rc = stream_device(static_cast<hipStream_t>(a->stream), &dev);
  if (rc != FORK_OK) return rc;
  void* ws = nullptr;
  rc = scratch_address(dev, &ws);
  if (rc != FORK_OK) return rc;
  return enqueue_step(a, ws, lay);
}

int fork_step(const void* hidden, const void* W_head, int32_t* tokens, uint8_t* mask,
              int32_t* block_start, int32_t block_len, float tau, float* out_conf,
              float* out_entropy, float* out_logp, int32_t* out_fallback, int32_t B, int32_t L,
              int32_t d, int32_t V, int32_t dtype, void* stream) {
  fork_step_args a = {};
  a.hidden = hidden;
  a.W_head = W_head;
  a.tokens = tokens;
  a.mask = mask;
  a.block_start = block_start;
  a.block_len = block_len;
  a.tau = tau;
  a.out_conf = out_conf;
  a.out_entropy = out_entropy;
  a.out_logp = out_logp;
  a.out_fallback = out_fallback;
  a.B = B;
  a.L = L;
  a.d = d;
  a.V = V;
  a.dtype = dtype;
  a.stream = stream;
  a.rule = FORK_RULE_LEFTMOST;
  return fork_step_ex(&a);
}

// fork_logprob workspace: [partials: nvt*n float4][target logits: n float].
static bool logprob_layout(int32_t n, int32_t V, size_t* zt_off, size_t* total) {
  if (n < 0 || V <= 0) return false;
  const size_t nvt = (size_t)fork::num_vocab_tiles(V);
  *zt_off = align_up(nvt * (size_t)n * sizeof(float4));
  *total = *zt_off + align_up((size_t)n * sizeof(float));
  return true;
}

size_t fork_logprob_workspace_bytes(int32_t n, int32_t V) {
  size_t zt, total;
  return logprob_layout(n, V, &zt, &total) ? total : 0;
}

int fork_logprob(const fork_logprob_args* a) {
  if (!a) return fail(FORK_EINVAL, "args is NULL");
  if (a->n < 0 || a->M <= 0 || a->d <= 0 || a->V <= 0)
    return fail(FORK_EINVAL, "sizes must be positive (n=%d M=%d d=%d V=%d)", a->n, a->M, a->d,
                a->V);
  if (a->dtype != FORK_BF16 && a->dtype != FORK_F32)
    return fail(FORK_EINVAL, "unknown dtype %d", a->dtype);
  if (!a->hidden || !a->W_head || (a->n > 0 && (!a->tokens || !a->out_logp)))
    return fail(FORK_EINVAL, "a required pointer is NULL");
  if (!a->rows && a->n > a->M)
    return fail(FORK_EINVAL, "without rows, n=%d entries need n <= M=%d", a->n, a->M);
  if (a->dtype == FORK_BF16 && a->d % 8 != 0)
    return fail(FORK_EUNSUPPORTED, "bf16 path needs d %% 8 == 0 (d=%d)", a->d);
  if (a->dtype == FORK_F32 && a->d % 4 != 0)
    return fail(FORK_EUNSUPPORTED, "fp32 path needs d %% 4 == 0 (d=%d)", a->d);
  if (a->d > kMaxD)
    return fail(FORK_EUNSUPPORTED, "d=%d exceeds the supported maximum %d", a->d, kMaxD);
  if (a->rows && (long long)a->M * a->d * (a->dtype == FORK_BF16 ? 2 : 4) >= (1LL << 31))
    return fail(FORK_EUNSUPPORTED, "gathered rows need M*d*element_size < 2^31");
  if (!grid_fits(a->n, a->V))
    return fail(FORK_EUNSUPPORTED, "n=%d entries x V=%d exceed one launch grid; split the batch",
                a->n, a->V);
  if (!aligned16(a->hidden) || !aligned16(a->W_head))
    return fail(FORK_EINVAL, "hidden and W_head must be 16-byte aligned");
  size_t zt_off, total;
  if (!logprob_layout(a->n, a->V, &zt_off, &total)) return fail(FORK_EINVAL, "invalid sizes");
  if (a->n == 0) return FORK_OK;
  void* ws = a->workspace;
  std::unique_lock<std::mutex> ws_lock;  // held until the launches are enqueued
  if (ws) {
    if (a->workspace_bytes < total)
      return fail(FORK_EINVAL, "workspace holds %zu bytes, %zu needed", a->workspace_bytes, total);
    if (((uintptr_t)ws % kAlign) != 0) return fail(FORK_EINVAL, "workspace must be 256-byte aligned");
  } else {
    int rc = get_workspace(static_cast<hipStream_t>(a->stream), total, &ws, &ws_lock);
    if (rc != FORK_OK) return rc;
  }
  float4* partials = static_cast<float4*>(ws);
  float* ztoken = reinterpret_cast<float*>(static_cast<char*>(ws) + zt_off);
  hipStream_t stream = static_cast<hipStream_t>(a->stream);
  const int nvt = fork::num_vocab_tiles(a->V);
  hipError_t e;
  if (a->ev_lmhead_begin) {
    e = hipEventRecord(static_cast<hipEvent_t>(a->ev_lmhead_begin), stream);
    if (e != hipSuccess) return fail(FORK_EHIP, "hipEventRecord: %s", hipGetErrorString(e));
  }
  e = fork::launch_gemm_stats(a->hidden, a->W_head, a->dtype == FORK_BF16, a->n, a->d, a->V,
                              partials, a->rows, a->M, fork::SampleArgs{},
                              fork::TargetArgs{a->tokens, ztoken}, stream);
  if (e != hipSuccess) return fail(FORK_EHIP, "gemm_stats launch: %s", hipGetErrorString(e));
  if (a->ev_lmhead_end) {
    e = hipEventRecord(static_cast<hipEvent_t>(a->ev_lmhead_end), stream);
    if (e != hipSuccess) return fail(FORK_EHIP, "hipEventRecord: %s", hipGetErrorString(e));
  }
  e = fork::launch_merge(partials, a->n, nvt, a->out_q, a->out_entropy, a->out_logp, a->out_lse,
                         nullptr, nullptr, nullptr, nullptr, a->tokens, ztoken, a->V, stream);
  if (e != hipSuccess) return fail(FORK_EHIP, "merge launch: %s", hipGetErrorString(e));
  return FORK_OK;
}

int fork_select(const fork_select_args* a) {
  if (!a) return fail(FORK_EINVAL, "args is NULL");
  if (a->B < 0 || a->L <= 0) return fail(FORK_EINVAL, "need B >= 0 and L > 0 (B=%d L=%d)", a->B, a->L);
  if (a->B > 0 && (!a->conf || !a->argmax || !a->tokens || !a->mask || !a->block_start ||
                   !a->out_fallback))
    return fail(FORK_EINVAL, "a required pointer is NULL");
  if ((long long)a->B * a->L > 0x7fffffffLL)
    return fail(FORK_EINVAL, "B*L = %lld does not fit int32", (long long)a->B * a->L);
  if (a->block_len <= 0 || a->block_len > a->L)
    return fail(FORK_EINVAL, "block_len=%d must lie in [1, L=%d]", a->block_len, a->L);
  if (!isfinite(a->tau)) return fail(FORK_EINVAL, "tau must be finite");
  if (a->rule < FORK_RULE_LEFTMOST || a->rule > FORK_RULE_RANDOM)
    return fail(FORK_EINVAL, "unknown fallback rule %d", a->rule);
  if (a->rule == FORK_RULE_RANDOM && a->B > 0 && !a->uniform)
    return fail(FORK_EINVAL, "FORK_RULE_RANDOM needs uniform");
  if (a->rule == FORK_RULE_MAXENT && a->B > 0 && !a->entropy)
    return fail(FORK_EINVAL, "FORK_RULE_MAXENT needs entropy");
  if (a->layout != FORK_LAYOUT_ROW_MAJOR && a->layout != FORK_LAYOUT_POSITION_MAJOR)
    return fail(FORK_EINVAL, "unknown layout %d", a->layout);
  if (a->B == 0) return FORK_OK;  // an empty batch: nothing to enqueue
  hipError_t e = fork::launch_select(a->B, a->L, a->block_len, a->tau, a->rule, a->conf,
                                     a->entropy, a->uniform, a->argmax, a->tokens, a->mask,
                                     a->block_start, a->out_fallback, a->out_ncommit,
                                     a->out_commit_pos, a->layout == FORK_LAYOUT_POSITION_MAJOR,
                                     static_cast<hipStream_t>(a->stream));
  if (e != hipSuccess) return fail(FORK_EHIP, "select launch: %s", hipGetErrorString(e));
  return FORK_OK;
}

int fork_grpo_objective(const fork_grpo_args* a) {
  if (!a) return fail(FORK_EINVAL, "args is NULL");
  if (a->n_groups < 0 || a->G <= 0 || a->n < 0)
    return fail(FORK_EINVAL, "sizes must be non-negative, G positive (n_groups=%d G=%d n=%d)",
                a->n_groups, a->G, a->n);
  if (a->G > fork::kMaxGroupSize)
    return fail(FORK_EINVAL, "G=%d exceeds the supported maximum %d", a->G, fork::kMaxGroupSize);
  if ((long long)a->n_groups * a->G > 0x7ffffffeLL) return fail(FORK_EINVAL, "too many rollouts");
  if (!(a->eps >= 0.0f) || !isfinite(a->eps))
    return fail(FORK_EINVAL, "eps must be finite and >= 0");
  if (!a->out_J || (a->n_groups > 0 && (!a->rewards || !a->offsets || !a->out_group_obj ||
                                         !a->out_skipped)) ||
      (a->n > 0 && (!a->lp_new || !a->lp_old)))
    return fail(FORK_EINVAL, "a required pointer is NULL");
  hipError_t e = fork::launch_grpo_objective(
      a->n_groups, a->G, a->n, a->rewards, a->offsets, a->lp_new, a->lp_old, a->eps, a->out_adv,
      a->out_ratio, a->out_term, a->out_rollout_obj, a->out_group_obj, a->out_skipped, a->out_J,
      static_cast<hipStream_t>(a->stream));
  if (e != hipSuccess) return fail(FORK_EHIP, "grpo launch: %s", hipGetErrorString(e));
  return FORK_OK;
}

int fork_top_entropy(const float* entropy, int32_t R, int32_t Lg, int32_t k, uint8_t* sel,
                     void* stream) {
  if (R < 0 || Lg <= 0 || k < 0 || k > Lg)
    return fail(FORK_EINVAL, "need R >= 0, Lg > 0, 0 <= k <= Lg (R=%d Lg=%d k=%d)", R, Lg, k);
  if (Lg > fork::kMaxTopEntropyLen)
    return fail(FORK_EUNSUPPORTED, "Lg=%d exceeds the supported maximum %d", Lg,
                fork::kMaxTopEntropyLen);
  if (R > 0 && (!entropy || !sel)) return fail(FORK_EINVAL, "a required pointer is NULL");
  hipError_t e = fork::launch_top_entropy(R, Lg, k, entropy, sel, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FORK_EHIP, "top_entropy launch: %s", hipGetErrorString(e));
  return FORK_OK;
}

size_t fork_workspace_bytes(int32_t B, int32_t L, int32_t V) {
  Layout lay;
  return layout_for(B, L, V, /*sampling=*/true, &lay) ? lay.total : 0;
}

const char* fork_last_error(void) { return g_err; }

void fork_release(void) { g_registry.release_all(); }

int fork_version(void) { return kVersion; }

}  // extern "C"
