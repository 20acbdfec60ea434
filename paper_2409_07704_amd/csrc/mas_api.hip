// libmas host entry points (C ABI declared in include/mas.h).
//
// Every entry point validates its arguments on the host, then only enqueues
// kernels on the caller's stream; nothing synchronises or copies to the host.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdlib.h>

#include <cmath>

#include <mutex>
#include <unordered_map>

#include "mas.h"
#include "mas_internal.h"

namespace mas {

static bool ws_ok(const void* ws, size_t bytes, const Layout& L) {
  return ws != nullptr && ((uintptr_t)ws % kAlign) == 0 && bytes >= L.bytes;
}

// Bound of every device-side wait, in polls without progress.  The
// MAS_WAIT_BOUND environment variable (a positive integer) replaces it: a
// diagnostic that lets tests drive the timeout path with small bounds.
static int32_t wait_bound() {
  const char* s = getenv("MAS_WAIT_BOUND");
  if (s && *s) {
    char* end = nullptr;
    const long v = strtol(s, &end, 10);
    if (end && *end == '\0' && v > 0 && v <= (1l << 30)) return (int32_t)v;
  }
  return kDefaultWaitBound;
}

// Words that carry a call's tag (flags, completion order, boundary hand-off
// words) are trusted once they hold the current call's tag.  Calls of one
// shape keep every region in place, so stale words only carry older tags;
// but a call of another shape lays the regions out elsewhere, over memory the
// previous call used for plain data (step masks, row starts), which may equal
// any tag.  So the tagged regions of the new layout are cleared, by a fill
// kernel on the call's stream, whenever a workspace is used with a shape
// other than the one of its previous call (mas_workspace_init leaves a
// workspace clear).
struct Shape {
  int32_t B, T, S;
};
static std::mutex g_ws_mu;
static std::unordered_map<uintptr_t, Shape> g_ws_shape;  // workspace -> shape of its last call (B = 0: clear)

static void note_clear_workspace(const void* ws) {
  std::lock_guard<std::mutex> lock(g_ws_mu);
  g_ws_shape[(uintptr_t)ws] = Shape{0, 0, 0};
}

static hipError_t prepare_workspace(void* ws, const Layout& L, hipStream_t stream) {
  std::lock_guard<std::mutex> lock(g_ws_mu);
  auto it = g_ws_shape.find((uintptr_t)ws);
  const bool clear = it != g_ws_shape.end() && it->second.B == 0;
  const bool same = it != g_ws_shape.end() && it->second.B == L.B && it->second.T == L.T && it->second.S == L.S;
  if (!clear && !same) {
    const hipError_t e = launch_fill(static_cast<char*>(ws) + L.off_done, L.off_pm - L.off_done, stream);
    if (e != hipSuccess) return e;
  }
  g_ws_shape[(uintptr_t)ws] = Shape{L.B, L.T, L.S};
  return hipSuccess;
}

static mas_status run(const float* value, const int32_t* t_x, const int32_t* t_y, const Layout& L,
                      int32_t* row_start, int32_t* durations, float* score, int32_t* status, uint8_t* path, void* ws,
                      hipStream_t stream, float sentinel = -INFINITY) {
  if (prepare_workspace(ws, L, stream) != hipSuccess) return MAS_ERR_HIP;
  char* base = static_cast<char*>(ws);
  KParams p;
  p.value = value;
  p.t_x = t_x;
  p.t_y = t_y;
  p.row_start = row_start;
  p.score = score;
  p.status = status;
  p.durations = durations;
  p.path = path;
  p.hdr = reinterpret_cast<WsHeader*>(base);
  p.done = reinterpret_cast<uint32_t*>(base + L.off_done);
  p.tmo = reinterpret_cast<uint32_t*>(base + L.off_tmo);
  p.order = reinterpret_cast<uint64_t*>(base + L.off_order);
  p.slots = reinterpret_cast<uint64_t*>(base + L.off_slots);
  p.pm = reinterpret_cast<uint32_t*>(base + L.off_pm);
  p.pd = reinterpret_cast<uint8_t*>(base + L.off_pd);
  p.B = L.B;
  p.T = L.T;
  p.S = L.S;
  p.NW = L.NW;
  p.NC = L.NC;
  p.EP = L.EP;
  p.NB = L.NB;
  p.ntile = (L.T + kPathTileRows - 1) / kPathTileRows;
  p.path16 = path && (L.S % 16 == 0) && ((uintptr_t)path % 16 == 0);
  p.spin_limit = wait_bound();
  p.neg = sentinel;
  p.legacy = std::isfinite(sentinel) ? 1 : 0;
  return launch_mas(p, stream) == hipSuccess ? MAS_OK : MAS_ERR_HIP;
}

// Workspace of mas_forward_static: one array per device, held until the
// process ends.  In host code `scratch` only names the symbol; its device
// address comes from hipGetSymbolAddress, once per device (scratch_ptr).
static __device__ __align__(256) uint8_t scratch[MAS_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch[kMaxDevices];  // device address of `scratch` per device, null until set up

// The current device's scratch address.  The first call on a device looks
// the address up and enqueues the array's initialisation (zeros and the
// workspace mark, by a fill kernel) on `stream`.
static mas_status scratch_ptr(hipStream_t stream, void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return MAS_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return MAS_ERR_HIP;
    if ((uintptr_t)ptr % kAlign != 0) return MAS_ERR_HIP;
    if (launch_ws_init(ptr, MAS_STATIC_SCRATCH_BYTES, stream) != hipSuccess) return MAS_ERR_HIP;
    note_clear_workspace(ptr);
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return MAS_OK;
}
}  // namespace mas

using namespace mas;

extern "C" {

size_t mas_workspace_bytes(int32_t B, int32_t T, int32_t S) {
  Layout L;
  return make_layout(B, T, S, &L) ? L.bytes : 0;
}

mas_status mas_workspace_init(void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!workspace) return MAS_ERR_NULL_POINTER;
  if ((uintptr_t)workspace % kAlign != 0 || workspace_bytes < sizeof(WsHeader) || workspace_bytes % 16 != 0)
    return MAS_ERR_WORKSPACE;
  if (launch_ws_init(workspace, workspace_bytes, stream) != hipSuccess) return MAS_ERR_HIP;
  note_clear_workspace(workspace);
  return MAS_OK;
}

mas_status mas_search(const float* value, const int32_t* t_x, const int32_t* t_y, int32_t B, int32_t T, int32_t S,
                      int32_t* row_start_out, int32_t* durations_out, float* score_out, int32_t* item_status_out,
                      void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!value || !t_x || !t_y || !row_start_out) return MAS_ERR_NULL_POINTER;
  Layout L;
  if (!make_layout(B, T, S, &L)) return MAS_ERR_BAD_SHAPE;
  if (!ws_ok(workspace, workspace_bytes, L)) return MAS_ERR_WORKSPACE;
  return run(value, t_x, t_y, L, row_start_out, durations_out, score_out, item_status_out, nullptr, workspace, stream);
}

mas_status mas_expand_path(const int32_t* row_start, int32_t B, int32_t T, int32_t S, uint8_t* path_out,
                           hipStream_t stream) {
  if (!row_start || !path_out) return MAS_ERR_NULL_POINTER;
  Layout L;
  if (!make_layout(B, T, S, &L)) return MAS_ERR_BAD_SHAPE;
  return launch_path(row_start, B, T, S, path_out, stream) == hipSuccess ? MAS_OK : MAS_ERR_HIP;
}

mas_status mas_expand_text(const void* text, const int32_t* row_start, int32_t B, int32_t T, int32_t S, int32_t C,
                           int32_t elem_bytes, void* out, hipStream_t stream) {
  if (!text || !row_start || !out) return MAS_ERR_NULL_POINTER;
  if (B < 1 || T < 1 || S < 1 || C < 1 || T > (1 << 30)) return MAS_ERR_BAD_SHAPE;
  if (elem_bytes != 1 && elem_bytes != 2 && elem_bytes != 4 && elem_bytes != 8) return MAS_ERR_BAD_SHAPE;
  const size_t row_bytes = (size_t)C * (size_t)elem_bytes;
  if (row_bytes > ((size_t)1 << 24)) return MAS_ERR_BAD_SHAPE;
  const double limit = 281474976710656.0;  // 2^48 bytes per tensor
  if ((double)B * (double)S * (double)row_bytes > limit || (double)B * (double)T * (double)row_bytes > limit)
    return MAS_ERR_BAD_SHAPE;
  return launch_text(text, row_start, B, T, S, row_bytes, out, stream) == hipSuccess ? MAS_OK : MAS_ERR_HIP;
}

mas_status mas_loglik(const float* mu, const float* log_sigma, const float* z, const int32_t* t_x, const int32_t* t_y,
                      int32_t B, int32_t T, int32_t S, int32_t D, float* value_out, hipStream_t stream) {
  if (!mu || !z || !t_x || !t_y || !value_out) return MAS_ERR_NULL_POINTER;
  Layout L;
  if (!make_layout(B, T, S, &L) || D < 1 || D > kLoglikMaxD) return MAS_ERR_BAD_SHAPE;
  return launch_loglik(mu, log_sigma, z, t_x, t_y, value_out, B, T, S, D, stream) == hipSuccess ? MAS_OK
                                                                                               : MAS_ERR_HIP;
}

mas_status mas_forward_ex(const float* value, const int32_t* t_x, const int32_t* t_y, uint8_t* path_out, int32_t B,
                          int32_t T, int32_t S, float* score_out, int32_t* item_status_out, void* workspace,
                          size_t workspace_bytes, hipStream_t stream) {
  if (!value || !t_x || !t_y || !path_out) return MAS_ERR_NULL_POINTER;
  Layout L;
  if (!make_layout(B, T, S, &L)) return MAS_ERR_BAD_SHAPE;
  if (!ws_ok(workspace, workspace_bytes, L)) return MAS_ERR_WORKSPACE;
  int32_t* rs = reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + L.off_rs);
  return run(value, t_x, t_y, L, rs, nullptr, score_out, item_status_out, path_out, workspace, stream);
}

mas_status mas_forward_sentinel(const float* value, const int32_t* t_x, const int32_t* t_y, uint8_t* path_out,
                                int32_t B, int32_t T, int32_t S, float sentinel, float* score_out,
                                int32_t* item_status_out, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!value || !t_x || !t_y || !path_out) return MAS_ERR_NULL_POINTER;
  if (!(sentinel < 0.0f) || !std::isfinite(sentinel)) return MAS_ERR_BAD_VALUE;
  Layout L;
  if (!make_layout(B, T, S, &L)) return MAS_ERR_BAD_SHAPE;
  if (!ws_ok(workspace, workspace_bytes, L)) return MAS_ERR_WORKSPACE;
  int32_t* rs = reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + L.off_rs);
  return run(value, t_x, t_y, L, rs, nullptr, score_out, item_status_out, path_out, workspace, stream, sentinel);
}

mas_status mas_forward(const float* value, const int32_t* t_x, const int32_t* t_y, uint8_t* path_out, int32_t B,
                       int32_t T, int32_t S, hipStream_t stream) {
  if (!value || !t_x || !t_y || !path_out) return MAS_ERR_NULL_POINTER;
  Layout L;
  if (!make_layout(B, T, S, &L)) return MAS_ERR_BAD_SHAPE;
  void* ws = nullptr;
  if (hipMallocAsync(&ws, L.bytes, stream) != hipSuccess) return MAS_ERR_HIP;
  mas_status s = mas_workspace_init(ws, L.bytes, stream);
  if (s == MAS_OK) s = mas_forward_ex(value, t_x, t_y, path_out, B, T, S, nullptr, nullptr, ws, L.bytes, stream);
  if (hipFreeAsync(ws, stream) != hipSuccess && s == MAS_OK) s = MAS_ERR_HIP;
  return s;
}

mas_status mas_forward_static(const float* value, const int32_t* t_x, const int32_t* t_y, uint8_t* path_out,
                              int32_t B, int32_t T, int32_t S, float* score_out, int32_t* item_status_out,
                              hipStream_t stream) {
  if (!value || !t_x || !t_y || !path_out) return MAS_ERR_NULL_POINTER;
  Layout L;
  if (!make_layout(B, T, S, &L)) return MAS_ERR_BAD_SHAPE;
  if (L.bytes > MAS_STATIC_SCRATCH_BYTES) return MAS_ERR_SCRATCH;
  void* ws = nullptr;
  const mas_status s = scratch_ptr(stream, &ws);
  if (s != MAS_OK) return s;
  int32_t* rs = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + L.off_rs);
  return run(value, t_x, t_y, L, rs, nullptr, score_out, item_status_out, path_out, ws, stream);
}

const char* mas_status_string(mas_status status) {
  switch (status) {
    case MAS_OK:
      return "MAS_OK";
    case MAS_ERR_NULL_POINTER:
      return "MAS_ERR_NULL_POINTER";
    case MAS_ERR_BAD_SHAPE:
      return "MAS_ERR_BAD_SHAPE";
    case MAS_ERR_WORKSPACE:
      return "MAS_ERR_WORKSPACE";
    case MAS_ERR_HIP:
      return "MAS_ERR_HIP";
    case MAS_ERR_SCRATCH:
      return "MAS_ERR_SCRATCH";
    case MAS_ERR_BAD_VALUE:
      return "MAS_ERR_BAD_VALUE";
  }
  return "MAS_ERR_UNKNOWN";
}

int mas_version(void) { return MAS_VERSION; }

}  // extern "C"
