// C ABI of the library: argument validation, per-device caches of feature
// tables and workspaces, and dispatch to the HIP kernels.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "kernels.hpp"
#include "prefill_blocks.hpp"
#include "prefill_mfma.hpp"
#include "sata.h"
#include "table.hpp"

namespace {

thread_local std::string g_last_error;

sata_status fail(sata_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

sata_status ok() {
  g_last_error.clear();
  return SATA_OK;
}

sata_status hip_fail(hipError_t e, const char* what) {
  return fail(SATA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

struct TableEntry {
  sata::FeatureTable host;
  uint64_t* packed = nullptr;
  float* weight = nullptr;
  uint32_t* gen = nullptr;
  std::vector<uint32_t> host_gen;
};

struct Workspace {
  void* ptr = nullptr;
  size_t bytes = 0;
};

struct DeviceCache {
  std::map<std::pair<int, int>, TableEntry> tables;
  std::map<hipStream_t, Workspace> workspaces;
  std::map<hipStream_t, Workspace> counters;  // zeroed at allocation; kernels leave them zero
};

std::mutex g_mu;
std::map<int, DeviceCache> g_devices;

// Upper bound on features per head accepted by the kernels.
constexpr int64_t kMaxFeatures = (int64_t)1 << 26;
// Upper bound on B*H (one grid dimension per head).
constexpr int kMaxHeads = 65535;
// Upper bound on the partial-readout workspace of one segment of a call.
constexpr size_t kMaxWorkspace = (size_t)512 << 20;
// The same for the generated-feature kernel, whose segments each store and
// reload the whole state (at d = 64 a 4096-token call of 16 heads is one
// segment).
constexpr size_t kMaxFeatWorkspace = (size_t)2 << 30;
// The same for the backward, whose scan workgroups load and store their state
// slice at every segment.
constexpr size_t kMaxBackwardWorkspace = (size_t)2 << 30;
// The tuned matrix-core kernels hold the partial readouts of the whole call;
// beyond this much the call takes the segmented kernels instead.
constexpr size_t kMaxWholeCallWorkspace = (size_t)4 << 30;
// The flat decode kernel (the one that takes residuals) serves d_v up to this.
constexpr int kMaxCompensatedDv = 127;

// Scratch of sata_decode_step_noalloc: one array per device for the life of
// the process.  The first kScratchCounterBytes hold the per-head arrival
// counters of the split decode (zeroed once per device by a fill kernel; the
// kernels set each counter back to zero), the rest the pieces' partial sums.
// In host code `scratch` names a host-side stand-in: only the address that
// hipGetSymbolAddress returns for the current device may reach a kernel.
constexpr size_t kScratchBytes = (size_t)4 << 20;
constexpr size_t kScratchCounterBytes = sizeof(int) * 65536;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

struct ScratchSlot {
  bool ready = false;
  unsigned char* ptr = nullptr;  // the device address of `scratch` on that device
};
constexpr int kMaxDevices = 64;
ScratchSlot g_scratch[kMaxDevices];  // guarded by g_mu

sata_status get_table(int d, int P, hipStream_t stream, sata::DevTable* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::lock_guard<std::mutex> lock(g_mu);
  DeviceCache& dc = g_devices[dev];
  auto key = std::make_pair(d, P);
  auto it = dc.tables.find(key);
  if (it == dc.tables.end()) {
    TableEntry ent;
    ent.host = sata::build_table(d, P);
    ent.host_gen = sata::build_gen_program(ent.host, sata::kTablePad, sata::kGenBlock);
    // the device copy ends in kTablePad zero entries
    ent.host.packed.resize(ent.host.packed.size() + sata::kTablePad, 0);
    ent.host.weight.resize(ent.host.weight.size() + sata::kTablePad, 0.0f);
    const size_t D = (size_t)ent.host.D + sata::kTablePad;
    auto release = [&ent]() {
      hipFree(ent.packed);
      hipFree(ent.weight);
      hipFree(ent.gen);
    };
    if ((e = hipMalloc(&ent.packed, D * sizeof(uint64_t))) != hipSuccess ||
        (e = hipMalloc(&ent.weight, D * sizeof(float))) != hipSuccess ||
        (e = hipMalloc(&ent.gen, 2 * D * sizeof(uint32_t))) != hipSuccess) {
      release();
      return hip_fail(e, "hipMalloc(table)");
    }
    // The host copies live in the cache, so asynchronous copies are safe.
    e = hipMemcpyAsync(ent.packed, ent.host.packed.data(), D * sizeof(uint64_t), hipMemcpyHostToDevice, stream);
    if (e == hipSuccess)
      e = hipMemcpyAsync(ent.weight, ent.host.weight.data(), D * sizeof(float), hipMemcpyHostToDevice, stream);
    if (e == hipSuccess)
      e = hipMemcpyAsync(ent.gen, ent.host_gen.data(), 2 * D * sizeof(uint32_t), hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) {
      release();
      return hip_fail(e, "uploading feature table");
    }
    it = dc.tables.emplace(key, std::move(ent)).first;
  }
  out->packed = it->second.packed;
  out->weight = it->second.weight;
  out->gen = it->second.gen;
  out->D = it->second.host.D;
  out->d = d;
  out->P = P;
  return SATA_OK;
}

// The cached table of (d, P) on the current device, without creating one.
sata_status find_table(int d, int P, sata::DevTable* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::lock_guard<std::mutex> lock(g_mu);
  auto dc = g_devices.find(dev);
  if (dc != g_devices.end()) {
    auto it = dc->second.tables.find(std::make_pair(d, P));
    if (it != dc->second.tables.end()) {
      out->packed = it->second.packed;
      out->weight = it->second.weight;
      out->gen = it->second.gen;
      out->D = it->second.host.D;
      out->d = d;
      out->P = P;
      return SATA_OK;
    }
  }
  return fail(SATA_ERR_UNSUPPORTED,
              "no feature table for d_k=%d P=%d on device %d yet: make one sata_decode_step, sata_prefill or "
              "sata_feature_map call with these sizes first",
              d, P, dev);
}

// The device address of `scratch` on the current device; on the first call
// on a device it is looked up and the counter region cleared on `stream`.
sata_status get_scratch(hipStream_t stream, unsigned char** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(SATA_ERR_UNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_mu);
  ScratchSlot& slot = g_scratch[dev];
  if (!slot.ready) {
    void* p = nullptr;
    if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess)
      return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if ((e = sata::launch_fill_zero((float*)p, (int64_t)(kScratchCounterBytes / sizeof(float)), stream)) !=
        hipSuccess)
      return hip_fail(e, "clearing the scratch counters");
    slot.ptr = (unsigned char*)p;
    slot.ready = true;
  }
  *out = slot.ptr;
  return SATA_OK;
}

// Returns a per-(device, stream) scratch buffer of at least `bytes`.
sata_status get_workspace(size_t bytes, hipStream_t stream, void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::lock_guard<std::mutex> lock(g_mu);
  Workspace& ws = g_devices[dev].workspaces[stream];
  if (ws.bytes < bytes) {
    if (ws.ptr) {
      // earlier work on this stream may still read the old buffer
      if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
      hipFree(ws.ptr);
      ws.ptr = nullptr;
      ws.bytes = 0;
    }
    size_t want = bytes < ((size_t)1 << 20) ? ((size_t)1 << 20) : bytes;
    if ((e = hipMalloc(&ws.ptr, want)) != hipSuccess) return hip_fail(e, "hipMalloc(workspace)");
    ws.bytes = want;
  }
  *out = ws.ptr;
  return SATA_OK;
}

// Returns a per-(device, stream) array of at least n ints, all zero.  It is
// cleared once, when allocated, by a fill kernel on the stream; the kernels
// that count in it set every counter back to zero.
sata_status get_counters(int64_t n, hipStream_t stream, int** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::lock_guard<std::mutex> lock(g_mu);
  Workspace& ws = g_devices[dev].counters[stream];
  const size_t bytes = sizeof(int) * (size_t)n;
  if (ws.bytes < bytes) {
    if (ws.ptr) {
      if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
      hipFree(ws.ptr);
      ws.ptr = nullptr;
      ws.bytes = 0;
    }
    size_t want = bytes < ((size_t)1 << 16) ? ((size_t)1 << 16) : bytes;
    if ((e = hipMalloc(&ws.ptr, want)) != hipSuccess) return hip_fail(e, "hipMalloc(counters)");
    if ((e = sata::launch_fill_zero((float*)ws.ptr, (int64_t)(want / sizeof(float)), stream)) != hipSuccess) {
      hipFree(ws.ptr);
      ws.ptr = nullptr;
      return hip_fail(e, "clearing counters");
    }
    ws.bytes = want;
  }
  *out = (int*)ws.ptr;
  return SATA_OK;
}

bool valid_dtype(sata_dtype t) { return t == SATA_F32 || t == SATA_BF16; }

sata_status check_dims(int d_k, int d_v, int P, int64_t* D) {
  if (d_k < 1 || d_k > sata::kMaxDim) return fail(SATA_ERR_INVALID_ARG, "d_k=%d outside 1..%d", d_k, sata::kMaxDim);
  if (d_v < 1 || d_v > sata::kMaxDim) return fail(SATA_ERR_INVALID_ARG, "d_v=%d outside 1..%d", d_v, sata::kMaxDim);
  if (P < 1 || P > sata::kMaxP) return fail(SATA_ERR_INVALID_ARG, "P=%d outside 1..%d", P, sata::kMaxP);
  const int64_t f = sata::feature_count(d_k, P);
  if (f < 0 || f > kMaxFeatures)
    return fail(SATA_ERR_TOO_LARGE, "C(d_k+P-1, P-1) features exceed %lld", (long long)kMaxFeatures);
  *D = f;
  return SATA_OK;
}

sata_status check_prefill_args(sata_dtype dt, int B, int H, int n, int d_k, int d_v, int P, int chunk,
                               int64_t* D) {
  if (!valid_dtype(dt)) return fail(SATA_ERR_INVALID_ARG, "unknown dtype %d", (int)dt);
  if (B < 1 || H < 1) return fail(SATA_ERR_INVALID_ARG, "B=%d H=%d must be >= 1", B, H);
  if (n < 0) return fail(SATA_ERR_INVALID_ARG, "n=%d < 0", n);
  sata_status st = check_dims(d_k, d_v, P, D);
  if (st != SATA_OK) return st;
  if (chunk != 16 && chunk != 32 && chunk != 64 && chunk != 128)
    return fail(SATA_ERR_UNSUPPORTED, "chunk=%d; supported: 16, 32, 64, 128", chunk);
  if ((int64_t)B * H > kMaxHeads) return fail(SATA_ERR_TOO_LARGE, "B*H=%lld exceeds %d", (long long)B * H, kMaxHeads);
  return SATA_OK;
}

enum class PrefillPath { kMfma32, kBlocks, kFeat, kFloat32 };

// The kernel family that serves a validated prefill request.
PrefillPath prefill_path(sata_dtype dt, int BH, int n, int d_k, int d_v, int P, int chunk) {
  sata::MfmaPrefillPlan mp;
  if (dt == SATA_BF16 && sata::plan_prefill_mfma(BH, n, d_k, d_v, P, chunk, &mp) &&
      mp.workspace_bytes <= kMaxWholeCallWorkspace)
    return PrefillPath::kMfma32;
  if (dt == SATA_BF16 && sata::plan_prefill_blocks(BH, n, d_k, d_v, P, chunk, &mp) &&
      mp.workspace_bytes <= kMaxWholeCallWorkspace)
    return PrefillPath::kBlocks;
  sata::FeatPrefillPlan fp;
  if (sata::plan_prefill_feat(sata::feature_count(d_k, P), BH, n, d_k, d_v, P, chunk, dt == SATA_F32, kMaxFeatWorkspace,
                              &fp))
    return PrefillPath::kFeat;
  return PrefillPath::kFloat32;
}

// One prefill over BH key/value heads; q and y hold qg query heads per
// key/value head (head bh's queries start at head bh * qg of q).
sata_status prefill_dispatch(const void* q, const void* k, const void* v, sata_dtype dt, int BH, int n, int d_k,
                             int d_v, int P, int chunk, void* y, float* S_out, hipStream_t s, int64_t D, int qg) {
  const int E = d_v + 1;
  hipError_t e;
  sata_status st;
  if (n == 0) {
    if (S_out) {
      if ((e = sata::launch_fill_zero(S_out, (int64_t)BH * D * E, s)) != hipSuccess)
        return hip_fail(e, "fill launch");
    }
    return ok();
  }
  sata::DevTable t;
  if ((st = get_table(d_k, P, s, &t)) != SATA_OK) return st;

  // bf16 fast path on the matrix cores where a tuned kernel exists
  sata::MfmaPrefillPlan mp;
  const PrefillPath path = prefill_path(dt, BH, n, d_k, d_v, P, chunk);
  if (path == PrefillPath::kMfma32 && sata::plan_prefill_mfma(BH, n, d_k, d_v, P, chunk, &mp)) {
    void* ws = nullptr;
    if ((st = get_workspace(mp.workspace_bytes, s, &ws)) != SATA_OK) return st;
    e = sata::launch_prefill_mfma(q, k, v, y, S_out, BH, n, d_k, d_v, P, chunk, mp, ws, s, qg);
    if (e != hipSuccess) return hip_fail(e, "prefill (matrix-core) launch");
    return ok();
  }
  if (path == PrefillPath::kBlocks && sata::plan_prefill_blocks(BH, n, d_k, d_v, P, chunk, &mp)) {
    void* ws = nullptr;
    if ((st = get_workspace(mp.workspace_bytes, s, &ws)) != SATA_OK) return st;
    e = sata::launch_prefill_blocks(q, k, v, y, S_out, BH, n, d_k, d_v, P, chunk, mp, ws, s, qg);
    if (e != hipSuccess) return hip_fail(e, "prefill (matrix-core, per-block) launch");
    return ok();
  }

  sata::FeatPrefillPlan fp;
  if (path == PrefillPath::kFeat &&
      sata::plan_prefill_feat(D, BH, n, d_k, d_v, P, chunk, dt == SATA_F32, kMaxFeatWorkspace, &fp)) {
    const size_t state_bytes = S_out ? 0 : sizeof(float) * (size_t)BH * D * E;
    void* ws = nullptr;
    if ((st = get_workspace(fp.partial_bytes + state_bytes, s, &ws)) != SATA_OK) return st;
    float* partial = (float*)ws;
    float* S_state = S_out ? S_out : (float*)((char*)ws + fp.partial_bytes);
    e = sata::launch_prefill_feat(q, k, v, y, BH, n, d_k, d_v, P, t, fp, S_state, partial, s, qg);
    if (e != hipSuccess) return hip_fail(e, "prefill (matrix-core, generated features) launch");
    return ok();
  }

  sata::PrefillGenericPlan plan;
  if (!sata::plan_prefill_generic(D, BH, n, d_k, d_v, chunk, kMaxWorkspace, &plan))
    return fail(SATA_ERR_UNSUPPORTED, "no slice size fits on chip for d_k=%d d_v=%d chunk=%d", d_k, d_v, chunk);
  const size_t state_bytes = S_out ? 0 : sizeof(float) * (size_t)BH * D * E;
  void* ws = nullptr;
  if ((st = get_workspace(plan.partial_bytes + state_bytes, s, &ws)) != SATA_OK) return st;
  float* partial = (float*)ws;
  float* S_state = S_out ? S_out : (float*)((char*)ws + plan.partial_bytes);
  e = sata::launch_prefill_generic(q, k, v, y, dt == SATA_BF16, BH, n, d_k, d_v, chunk, t, plan, S_state,
                                   partial, s, qg);
  if (e != hipSuccess) return hip_fail(e, "prefill launch");
  return ok();
}

sata_status decode_step(float* S, float* R, const void* q, const void* k, const void* v, sata_dtype dt, int B,
                        int H, int d_k, int d_v, int P, void* y, void* stream) {
  if (!valid_dtype(dt)) return fail(SATA_ERR_INVALID_ARG, "unknown dtype %d", (int)dt);
  if (B < 1 || H < 1) return fail(SATA_ERR_INVALID_ARG, "B=%d H=%d must be >= 1", B, H);
  int64_t D = 0;
  sata_status st = check_dims(d_k, d_v, P, &D);
  if (st != SATA_OK) return st;
  if ((int64_t)B * H > kMaxHeads) return fail(SATA_ERR_TOO_LARGE, "B*H=%lld exceeds %d", (long long)B * H, kMaxHeads);
  if (!S || !q || !k || !v || !y) return fail(SATA_ERR_INVALID_ARG, "null tensor pointer");
  const int BH = B * H;
  hipStream_t s = (hipStream_t)stream;
  sata::DecodePlan plan = sata::plan_decode(D, d_k, d_v, BH);
  if (R && !sata::decode_supports_residuals(plan, S))
    return fail(SATA_ERR_UNSUPPORTED, "the compensated decode needs a 16-byte aligned state and d_v <= %d",
                kMaxCompensatedDv);
  sata::DevTable t;
  if ((st = get_table(d_k, P, s, &t)) != SATA_OK) return st;
  float* partial = nullptr;
  int* counters = nullptr;
  // partial sums: one row per slice (row-wise path) or per piece of a head (flat path)
  const int64_t rows = std::max<int64_t>(plan.nslices > 1 ? plan.nslices : 0, plan.flat_np > 1 ? plan.flat_np : 0);
  if (rows > 0) {
    void* ws = nullptr;
    const size_t bytes = sizeof(float) * (size_t)BH * rows * (d_v + 1);
    if ((st = get_workspace(bytes, s, &ws)) != SATA_OK) return st;
    partial = (float*)ws;
  }
  if (plan.flat_np > 1 && (st = get_counters(BH, s, &counters)) != SATA_OK) return st;
  hipError_t e =
      sata::launch_decode(S, q, k, v, y, dt == SATA_BF16, BH, d_k, d_v, t, plan, partial, counters, s, R);
  if (e != hipSuccess) return hip_fail(e, "decode launch");
  return ok();
}

}  // namespace

extern "C" {

int64_t sata_feature_count(int d, int P) {
  if (d < 1 || P < 1) return -1;
  return sata::feature_count(d, P);
}

int64_t sata_state_elems(int d_k, int d_v, int P) {
  if (d_k < 1 || d_v < 1 || P < 1) return -1;
  const int64_t f = sata::feature_count(d_k, P);
  if (f < 0 || f > INT64_MAX / (d_v + 1)) return -1;
  return f * (d_v + 1);
}

sata_status sata_feature_index(int d, int P, int64_t f, int* degree, int* idx) {
  if (!degree || !idx) return fail(SATA_ERR_INVALID_ARG, "null output pointer");
  if (d < 1 || d > sata::kMaxDim || P < 1 || P > sata::kMaxP)
    return fail(SATA_ERR_INVALID_ARG, "d=%d or P=%d out of range", d, P);
  const int64_t D = sata::feature_count(d, P);
  if (D < 0 || f < 0 || f >= D) return fail(SATA_ERR_INVALID_ARG, "feature %lld out of range", (long long)f);
  // skip whole degrees, then walk the tuples of the degree that holds f
  int64_t base = 0;
  for (int p = 0; p < P; ++p) {
    const int64_t m = sata::binom((int64_t)d + p - 1, p);
    if (f < base + m) {
      int64_t i = base;
      bool found = false;
      if (p == 0) found = true;
      else
        sata::for_each_tuple(d, p, [&](const int* t) {
          if (!found && i == f) {
            for (int j = 0; j < p; ++j) idx[j] = t[j];
            found = true;
          }
          ++i;
        });
      *degree = p;
      return ok();
    }
    base += m;
  }
  return fail(SATA_ERR_INVALID_ARG, "feature %lld out of range", (long long)f);
}

sata_status sata_feature_map(const void* x, sata_dtype xt, int64_t rows, int d, int P, float* phi,
                             void* stream) {
  if (!valid_dtype(xt)) return fail(SATA_ERR_INVALID_ARG, "unknown dtype %d", (int)xt);
  if (rows < 0) return fail(SATA_ERR_INVALID_ARG, "rows=%lld < 0", (long long)rows);
  int64_t D = 0;
  sata_status st = check_dims(d, 1, P, &D);
  if (st != SATA_OK) return st;
  if (rows == 0) return ok();
  if (!x || !phi) return fail(SATA_ERR_INVALID_ARG, "null tensor pointer");
  hipStream_t s = (hipStream_t)stream;
  sata::DevTable t;
  if ((st = get_table(d, P, s, &t)) != SATA_OK) return st;
  hipError_t e = sata::launch_feature_map(x, xt == SATA_BF16, rows, t, phi, s);
  if (e != hipSuccess) return hip_fail(e, "feature_map launch");
  return ok();
}

sata_status sata_prefill_operands(sata_dtype dt, int B, int H, int n, int d_k, int d_v, int P, int chunk,
                                  sata_operands* operands) {
  if (!operands) return fail(SATA_ERR_INVALID_ARG, "null output pointer");
  int64_t D = 0;
  sata_status st = check_prefill_args(dt, B, H, n, d_k, d_v, P, chunk, &D);
  if (st != SATA_OK) return st;
  if (prefill_path(dt, B * H, n, d_k, d_v, P, chunk) == PrefillPath::kFloat32)
    *operands = SATA_OPERANDS_F32;
  else
    *operands = dt == SATA_BF16 ? SATA_OPERANDS_BF16 : SATA_OPERANDS_SPLIT;
  return ok();
}

sata_status sata_prefill_parts(sata_dtype dt, int B, int H, int n, int d_k, int d_v, int P, int chunk, int* parts) {
  if (!parts) return fail(SATA_ERR_INVALID_ARG, "null output pointer");
  int64_t D = 0;
  sata_status st = check_prefill_args(dt, B, H, n, d_k, d_v, P, chunk, &D);
  if (st != SATA_OK) return st;
  *parts = 1;
  sata::FeatPrefillPlan fp;
  if (prefill_path(dt, B * H, n, d_k, d_v, P, chunk) == PrefillPath::kFeat &&
      sata::plan_prefill_feat(D, B * H, n, d_k, d_v, P, chunk, dt == SATA_F32, kMaxFeatWorkspace, &fp))
    *parts = fp.parts;
  return ok();
}

sata_status sata_prefill(const void* q, const void* k, const void* v, sata_dtype dt, int B, int H, int n,
                         int d_k, int d_v, int P, int chunk, void* y, float* S_out, void* stream) {
  int64_t D = 0;
  sata_status st = check_prefill_args(dt, B, H, n, d_k, d_v, P, chunk, &D);
  if (st != SATA_OK) return st;
  if (n > 0 && (!q || !k || !v || !y)) return fail(SATA_ERR_INVALID_ARG, "null tensor pointer");
  return prefill_dispatch(q, k, v, dt, B * H, n, d_k, d_v, P, chunk, y, S_out, (hipStream_t)stream, D, 1);
}

sata_status sata_prefill_grouped(const void* q, const void* k, const void* v, sata_dtype dt, int B, int H_kv,
                                 int G, int n, int d_k, int d_v, int P, int chunk, void* y, float* S_out,
                                 void* stream) {
  if (G < 1) return fail(SATA_ERR_INVALID_ARG, "G=%d must be >= 1", G);
  if (B >= 1 && H_kv >= 1 && (int64_t)B * H_kv * G > kMaxHeads)
    return fail(SATA_ERR_TOO_LARGE, "B*H_kv*G=%lld exceeds %d", (long long)B * H_kv * G, kMaxHeads);
  int64_t D = 0;
  sata_status st = check_prefill_args(dt, B, H_kv, n, d_k, d_v, P, chunk, &D);
  if (st != SATA_OK) return st;
  if (n > 0 && (!q || !k || !v || !y)) return fail(SATA_ERR_INVALID_ARG, "null tensor pointer");
  const size_t esz = dt == SATA_BF16 ? 2 : 4;
  // query head g + G h of each batch row is member g of key/value head h's
  // group: with the heads of the call numbered by key/value head, member g's
  // queries and outputs start g heads in and lie G heads apart
  for (int g = 0; g < G; ++g) {
    const void* qg = (const char*)q + esz * (size_t)g * (size_t)n * (size_t)d_k;
    void* yg = (char*)y + esz * (size_t)g * (size_t)n * (size_t)d_v;
    st = prefill_dispatch(qg, k, v, dt, B * H_kv, n, d_k, d_v, P, chunk, yg, g == 0 ? S_out : nullptr,
                          (hipStream_t)stream, D, G);
    if (st != SATA_OK) return st;
    if (n == 0) break;
  }
  return ok();
}

sata_status sata_backward(const void* q, const void* k, const void* v, const void* dy, sata_dtype dt, int B, int H,
                          int n, int d_k, int d_v, int P, int chunk, void* dq, void* dk, void* dv, void* stream) {
  if (!valid_dtype(dt)) return fail(SATA_ERR_INVALID_ARG, "unknown dtype %d", (int)dt);
  if (B < 1 || H < 1) return fail(SATA_ERR_INVALID_ARG, "B=%d H=%d must be >= 1", B, H);
  if (n < 0) return fail(SATA_ERR_INVALID_ARG, "n=%d < 0", n);
  int64_t D = 0;
  sata_status st = check_dims(d_k, d_v, P, &D);
  if (st != SATA_OK) return st;
  if ((int64_t)B * H > kMaxHeads) return fail(SATA_ERR_TOO_LARGE, "B*H=%lld exceeds %d", (long long)B * H, kMaxHeads);
  if (chunk != 16 && chunk != 32 && chunk != 64)
    return fail(SATA_ERR_UNSUPPORTED, "chunk=%d; the backward supports 16, 32, 64", chunk);
  if (d_k > sata::kMaxBackwardDim || d_v > sata::kMaxBackwardDim)
    return fail(SATA_ERR_UNSUPPORTED, "the backward supports d_k, d_v <= %d", sata::kMaxBackwardDim);
  if (n == 0) return ok();
  if (!q || !k || !v || !dy || !dq || !dk || !dv) return fail(SATA_ERR_INVALID_ARG, "null tensor pointer");
  const int BH = B * H;
  sata::BackwardPlan plan;
  sata::PrefillGenericPlan fwd;
  if (!sata::plan_backward(D, BH, n, d_k, d_v, P, chunk, kMaxBackwardWorkspace, &plan, &fwd))
    return fail(SATA_ERR_UNSUPPORTED, "no backward slice fits on chip for d_k=%d d_v=%d chunk=%d", d_k, d_v, chunk);
  hipStream_t s = (hipStream_t)stream;
  sata::DevTable t;
  if ((st = get_table(d_k, P, s, &t)) != SATA_OK) return st;
  void* ws = nullptr;
  if ((st = get_workspace(plan.h_bytes + plan.state_bytes + plan.partial_bytes, s, &ws)) != SATA_OK) return st;
  float* h = (float*)ws;
  float* state = (float*)((char*)ws + plan.h_bytes);
  float* partial = (float*)((char*)ws + plan.h_bytes + plan.state_bytes);
  hipError_t e = sata::launch_backward(q, k, v, dy, dq, dk, dv, dt == SATA_BF16, BH, n, d_k, d_v, P, chunk, t, plan,
                                       fwd, h, state, partial, s);
  if (e != hipSuccess) return hip_fail(e, "backward launch");
  return ok();
}

sata_status sata_decode_step(float* S, const void* q, const void* k, const void* v, sata_dtype dt, int B,
                             int H, int d_k, int d_v, int P, void* y, void* stream) {
  return decode_step(S, nullptr, q, k, v, dt, B, H, d_k, d_v, P, y, stream);
}

sata_status sata_decode_step_noalloc(float* S, const void* q, const void* k, const void* v, sata_dtype dt, int B,
                                    int H, int d_k, int d_v, int P, void* y, void* stream) {
  if (!valid_dtype(dt)) return fail(SATA_ERR_INVALID_ARG, "unknown dtype %d", (int)dt);
  if (B < 1 || H < 1) return fail(SATA_ERR_INVALID_ARG, "B=%d H=%d must be >= 1", B, H);
  int64_t D = 0;
  sata_status st = check_dims(d_k, d_v, P, &D);
  if (st != SATA_OK) return st;
  if ((int64_t)B * H > kMaxHeads) return fail(SATA_ERR_TOO_LARGE, "B*H=%lld exceeds %d", (long long)B * H, kMaxHeads);
  if (!S || !q || !k || !v || !y) return fail(SATA_ERR_INVALID_ARG, "null tensor pointer");
  const int BH = B * H;
  sata::DecodePlan plan = sata::plan_decode(D, d_k, d_v, BH);
  const int64_t rows = std::max<int64_t>(plan.nslices > 1 ? plan.nslices : 0, plan.flat_np > 1 ? plan.flat_np : 0);
  const size_t partial_bytes = sizeof(float) * (size_t)BH * (size_t)rows * (size_t)(d_v + 1);
  if (partial_bytes > kScratchBytes - kScratchCounterBytes)
    return fail(SATA_ERR_TOO_LARGE, "partial sums of %zu bytes exceed the %zu-byte scratch", partial_bytes,
                kScratchBytes - kScratchCounterBytes);
  sata::DevTable t;
  if ((st = find_table(d_k, P, &t)) != SATA_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  unsigned char* base = nullptr;
  if ((st = get_scratch(s, &base)) != SATA_OK) return st;
  float* partial = rows > 0 ? (float*)(base + kScratchCounterBytes) : nullptr;
  int* counters = plan.flat_np > 1 ? (int*)base : nullptr;
  hipError_t e = sata::launch_decode(S, q, k, v, y, dt == SATA_BF16, BH, d_k, d_v, t, plan, partial, counters, s);
  if (e != hipSuccess) return hip_fail(e, "decode launch");
  return ok();
}

sata_status sata_decode_step_compensated(float* S, float* R, const void* q, const void* k, const void* v,
                                         sata_dtype dt, int B, int H, int d_k, int d_v, int P, void* y,
                                         void* stream) {
  if (!R) return fail(SATA_ERR_INVALID_ARG, "null residual pointer");
  return decode_step(S, R, q, k, v, dt, B, H, d_k, d_v, P, y, stream);
}

int64_t sata_residual_elems(int d_k, int d_v, int P) {
  if (d_k < 1 || d_v < 1 || P < 1) return -1;
  const int64_t f = sata::feature_count(d_k, P);
  if (f < 0) return -1;
  return f + (int64_t)(d_k + 1) * d_v;
}

sata_status sata_decode_step_grouped(float* S, const void* q, const void* k, const void* v, sata_dtype dt, int B,
                                     int H_kv, int G, int d_k, int d_v, int P, void* y, void* stream) {
  if (!valid_dtype(dt)) return fail(SATA_ERR_INVALID_ARG, "unknown dtype %d", (int)dt);
  if (B < 1 || H_kv < 1) return fail(SATA_ERR_INVALID_ARG, "B=%d H_kv=%d must be >= 1", B, H_kv);
  if (G < 1) return fail(SATA_ERR_INVALID_ARG, "G=%d must be >= 1", G);
  int64_t D = 0;
  sata_status st = check_dims(d_k, d_v, P, &D);
  if (st != SATA_OK) return st;
  if ((int64_t)B * H_kv * G > kMaxHeads)
    return fail(SATA_ERR_TOO_LARGE, "B*H_kv*G=%lld exceeds %d", (long long)B * H_kv * G, kMaxHeads);
  if (!S || !q || !k || !v || !y) return fail(SATA_ERR_INVALID_ARG, "null tensor pointer");
  if (G == 1) return sata_decode_step(S, q, k, v, dt, B, H_kv, d_k, d_v, P, y, stream);
  if (G != 2 && G != 4 && G != 8) return fail(SATA_ERR_UNSUPPORTED, "G=%d; supported: 1, 2, 4, 8", G);
  if (((uintptr_t)S & 15) != 0) return fail(SATA_ERR_UNSUPPORTED, "grouped decode needs a 16-byte aligned state");
  const int BH = B * H_kv;
  sata::GroupedDecodePlan plan = sata::plan_decode_grouped(D, d_k, d_v, BH, G);
  if (plan.tu <= 0)
    return fail(SATA_ERR_UNSUPPORTED, "no grouped decode plan fits on chip for d_k=%d d_v=%d P=%d G=%d", d_k, d_v, P,
                G);
  hipStream_t s = (hipStream_t)stream;
  sata::DevTable t;
  if ((st = get_table(d_k, P, s, &t)) != SATA_OK) return st;
  float* partial = nullptr;
  int* counters = nullptr;
  if (plan.np > 1) {
    void* ws = nullptr;
    const size_t bytes = sizeof(float) * (size_t)BH * plan.np * G * (d_v + 1);
    if ((st = get_workspace(bytes, s, &ws)) != SATA_OK) return st;
    partial = (float*)ws;
    if ((st = get_counters(BH, s, &counters)) != SATA_OK) return st;
  }
  hipError_t e = sata::launch_decode_grouped(S, q, k, v, y, dt == SATA_BF16, BH, d_k, d_v, t, plan, partial,
                                             counters, s);
  if (e != hipSuccess) return hip_fail(e, "grouped decode launch");
  return ok();
}

const char* sata_status_string(sata_status s) {
  switch (s) {
    case SATA_OK: return "ok";
    case SATA_ERR_INVALID_ARG: return "invalid argument";
    case SATA_ERR_UNSUPPORTED: return "unsupported";
    case SATA_ERR_TOO_LARGE: return "too large";
    case SATA_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}

const char* sata_last_error(void) { return g_last_error.c_str(); }

void sata_release(void) {
  std::lock_guard<std::mutex> lock(g_mu);
  int cur = 0;
  hipGetDevice(&cur);
  for (auto& kv : g_devices) {
    hipSetDevice(kv.first);
    for (auto& t : kv.second.tables) {
      hipFree(t.second.packed);
      hipFree(t.second.weight);
      hipFree(t.second.gen);
    }
    for (auto& w : kv.second.workspaces) hipFree(w.second.ptr);
    for (auto& w : kv.second.counters) hipFree(w.second.ptr);
  }
  g_devices.clear();
  hipSetDevice(cur);
}

}  // extern "C"
