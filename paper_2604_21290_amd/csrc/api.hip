// Host side of the C ABI declared in include/graphleap.h: argument checks,
// kernel dispatch and the lookahead schedule (Sec. III, Sec. IV-A/F).
#include <stdarg.h>
#include <stdio.h>

#include <climits>
#include <initializer_list>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "graphleap.h"
#include "gl_kernels.h"

namespace {

thread_local std::string g_last_error;

gl_status fail(gl_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

gl_status hip_fail(hipError_t e, const char* what) {
  return fail(GL_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

size_t esize(gl_dtype dt) { return dt == GL_BF16 ? 2 : 4; }
int vec_width(gl_dtype dt) { return dt == GL_BF16 ? 8 : 4; }
bool dtype_ok(gl_dtype dt) { return dt == GL_F32 || dt == GL_BF16; }
bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
  return a0 < b0 + nb && b0 < a0 + na;
}

// Tensors must be indexable with the kernels' 32-bit row counters.
bool size_ok(long long a, long long b, long long c) {
  const long long r = a * b;
  return a > 0 && b > 0 && c > 0 && r <= INT_MAX && r * c <= (1LL << 40);
}

gl_status check_knn(const void* x, int B, int N, int C, const void* keys, int M, int k, int dil,
                    gl_dtype dt, const int32_t* idx_out) {
  if (!x || !idx_out) return fail(GL_ERR_NULL_PTR, "knn: x and idx_out are required");
  if (!dtype_ok(dt)) return fail(GL_ERR_UNSUPPORTED, "knn: unknown dtype %d", (int)dt);
  if (B < 1 || N < 1 || C < 1 || B > 65535 || !size_ok(B, N, C))
    return fail(GL_ERR_BAD_SHAPE, "knn: bad shape B=%d N=%d C=%d", B, N, C);
  if (!keys && M != N) return fail(GL_ERR_BAD_SHAPE, "knn: keys=NULL needs M == N (M=%d N=%d)", M, N);
  if (M < 1 || M > GL_MAX_M || !size_ok(B, M, C))
    return fail(GL_ERR_BAD_SHAPE, "knn: M=%d outside [1, %d]", M, GL_MAX_M);
  if (C % vec_width(dt))
    return fail(GL_ERR_UNSUPPORTED, "knn: C=%d must be a multiple of %d", C, vec_width(dt));
  if (k < 1 || dil < 1 || (long long)k * dil > M || (long long)k * dil > GL_MAX_KD)
    return fail(GL_ERR_BAD_K, "knn: need 1<=k, 1<=dilation, k*dilation <= min(M=%d, %d); got k=%d d=%d",
                M, GL_MAX_KD, k, dil);
  if (gl::knn_smem_bytes(C, dt == GL_BF16) > 160 * 1024)
    return fail(GL_ERR_UNSUPPORTED, "knn: C=%d too wide for the LDS query tile", C);
  if (!aligned(x, 16) || (keys && !aligned(keys, 16)) || !aligned(idx_out, 4))
    return fail(GL_ERR_ALIGNMENT, "knn: x/keys need 16-byte, idx_out 4-byte alignment");
  const size_t ib = (size_t)B * N * k * 4, xb = (size_t)B * N * C * esize(dt),
               kb = keys ? (size_t)B * M * C * esize(dt) : 0;
  if (overlap(idx_out, ib, x, xb) || overlap(idx_out, ib, keys, kb))
    return fail(GL_ERR_ALIAS, "knn: idx_out overlaps x or keys");
  return GL_OK;
}

gl_status check_pool(const void* x, int B, int H, int W, int C, int r, gl_dtype dt,
                     const void* keys_out) {
  if (!x || !keys_out) return fail(GL_ERR_NULL_PTR, "pool: x and keys_out are required");
  if (!dtype_ok(dt)) return fail(GL_ERR_UNSUPPORTED, "pool: unknown dtype %d", (int)dt);
  if (B < 1 || H < 1 || W < 1 || C < 1 || r < 1 || H % r || W % r || !size_ok(B, (long long)H * W, C))
    return fail(GL_ERR_BAD_SHAPE, "pool: bad shape B=%d H=%d W=%d C=%d r=%d", B, H, W, C, r);
  if (C % vec_width(dt))
    return fail(GL_ERR_UNSUPPORTED, "pool: C=%d must be a multiple of %d", C, vec_width(dt));
  if (!aligned(x, 16) || !aligned(keys_out, 16))
    return fail(GL_ERR_ALIGNMENT, "pool: x/keys_out need 16-byte alignment");
  const size_t xb = (size_t)B * H * W * C * esize(dt);
  const size_t kb = (size_t)B * (H / r) * (W / r) * C * esize(dt);
  if (overlap(x, xb, keys_out, kb)) return fail(GL_ERR_ALIAS, "pool: keys_out overlaps x");
  return GL_OK;
}

// Row tiles of the fused MRConv tile (0: the tile does not fit LDS).
int mrconv_rt(int C, int k, gl_dtype dt) {
  const int dtb = dt == GL_BF16;
  const int rt = gl::mrconv_row_tiles(C, k, dtb, 65536);
  return rt ? rt : gl::mrconv_row_tiles(C, k, dtb, 160 * 1024);
}

gl_status check_mrconv(const void* x, int B, int N, int C, const void* keys, int M,
                       const int32_t* idx, int k, const void* W, const void* bias, int Cout,
                       gl_dtype dt, const void* out, int* rt_out, size_t w_bytes = 0) {
  if (!x || !idx || !W || !out) return fail(GL_ERR_NULL_PTR, "mrconv: x, idx, W and out are required");
  if (!dtype_ok(dt)) return fail(GL_ERR_UNSUPPORTED, "mrconv: unknown dtype %d", (int)dt);
  if (B < 1 || N < 1 || C < 1 || Cout < 1 || !size_ok(B, N, C) || !size_ok(B, N, Cout))
    return fail(GL_ERR_BAD_SHAPE, "mrconv: bad shape B=%d N=%d C=%d Cout=%d", B, N, C, Cout);
  if (!keys && M != N) return fail(GL_ERR_BAD_SHAPE, "mrconv: keys=NULL needs M == N");
  if (M < 1 || !size_ok(B, M, C)) return fail(GL_ERR_BAD_SHAPE, "mrconv: bad M=%d", M);
  if (k < 1 || k > GL_MAX_K) return fail(GL_ERR_BAD_K, "mrconv: k=%d outside [1, %d]", k, GL_MAX_K);
  if (C % vec_width(dt))
    return fail(GL_ERR_UNSUPPORTED, "mrconv: C=%d must be a multiple of %d", C, vec_width(dt));
  // the kernels address a neighbour row by its offset in 16-byte vectors (int32)
  if ((long long)M * (C / vec_width(dt)) > INT_MAX)
    return fail(GL_ERR_BAD_SHAPE, "mrconv: M=%d rows of C=%d exceed 2^31 16-byte vectors per image", M, C);
  // rt = 0: the fused LDS tile does not fit; the two-pass form is used
  const int rt = mrconv_rt(C, k, dt);
  if (!aligned(x, 16) || (keys && !aligned(keys, 16)) || !aligned(W, 16) || !aligned(out, 16) ||
      !aligned(idx, 4) || (bias && !aligned(bias, esize(dt))))
    return fail(GL_ERR_ALIGNMENT, "mrconv: x/keys/W/out need 16-byte alignment");
  const size_t es = esize(dt);
  const size_t ob = (size_t)B * N * Cout * es;
  if (!w_bytes) w_bytes = (size_t)Cout * 2 * C * es;
  if (overlap(out, ob, x, (size_t)B * N * C * es) ||
      overlap(out, ob, keys, keys ? (size_t)B * M * C * es : 0) ||
      overlap(out, ob, idx, (size_t)B * N * k * 4) || overlap(out, ob, W, w_bytes) ||
      overlap(out, ob, bias, bias ? (size_t)Cout * es : 0))
    return fail(GL_ERR_ALIAS, "mrconv: out overlaps an input");
  if (rt_out) *rt_out = rt;
  return GL_OK;
}

// Workspace bytes of one MRConv (the [x | m] rows of the two-pass form; 0 for
// the fused tile).
size_t mrconv_ws_need(int B, int N, int C, int k, int Cout, gl_dtype dt, int rt) {
  const int dtb = dt == GL_BF16;
  return gl::mrconv_use_split(C, Cout, dtb, rt, B * N) ? gl::mrconv_split_ws_bytes(B * N, C, dtb) : 0;
}

// A caller workspace of `need` bytes: present, large enough, 16-byte aligned,
// and (when given) clear of the call's other buffers.
gl_status check_ws(const char* who, size_t need, const void* ws, size_t ws_bytes,
                   std::initializer_list<std::pair<const void*, size_t>> others = {}) {
  if (need == 0) return GL_OK;
  if (!ws || ws_bytes < need)
    return fail(GL_ERR_WORKSPACE, "%s: needs a workspace of %zu bytes (got %zu at %p)", who, need,
                ws ? ws_bytes : (size_t)0, ws);
  if (!aligned(ws, 16)) return fail(GL_ERR_WORKSPACE, "%s: workspace must be 16-byte aligned", who);
  for (const auto& o : others)
    if (overlap(ws, need, o.first, o.second))
      return fail(GL_ERR_ALIAS, "%s: workspace overlaps another argument", who);
  return GL_OK;
}

constexpr uint32_t kHandleMagic = 0x474c4c41u;  // "GLLA"

}  // namespace

struct gl_lookahead {
  uint32_t magic;
  hipStream_t su, sb;
  hipEvent_t ev_ready, ev_built;
  bool pending;
  int prof_max;
  int prof_n[4];                                           // builds, updates, fused, linear
  std::vector<std::pair<hipEvent_t, hipEvent_t>> prof[4];
};

namespace {

bool handle_ok(gl_lookahead_t h) { return h && h->magic == kHandleMagic; }

// The MRConv workspace of one block of the handle's schedules: the caller's
// (already checked to be large enough), or null when the fused tile is used.
void* block_ws(int B, int N, int C, int k, gl_dtype dt, int rt, void* ws) {
  return mrconv_ws_need(B, N, C, k, C, dt, rt) ? ws : nullptr;
}

void free_profiling(gl_lookahead_t h) {
  for (int w = 0; w < 4; ++w) {
    for (auto& p : h->prof[w]) {
      (void)hipEventDestroy(p.first);
      (void)hipEventDestroy(p.second);
    }
    h->prof[w].clear();
    h->prof_n[w] = 0;
  }
  h->prof_max = 0;
}

// One launch, stamped with a pair of profiling events when enabled
// (which: 0 build, 1 update).  The events are recorded by the dispatch itself.
template <class Launch>
gl_status timed_launch(gl_lookahead_t h, int which, const char* what, Launch&& launch) {
  const int i = h->prof_n[which];
  const bool prof = i < h->prof_max;
  hipEvent_t e0 = prof ? h->prof[which][i].first : nullptr;
  hipEvent_t e1 = prof ? h->prof[which][i].second : nullptr;
  hipError_t e = launch(e0, e1);
  if (e != hipSuccess) return hip_fail(e, what);
  if (prof) h->prof_n[which] = i + 1;
  return GL_OK;
}

// kNN build on the build stream.
gl_status enqueue_build(gl_lookahead_t h, const void* x, int B, int N, int C, const void* keys,
                        int M, int k, int dil, gl_dtype dt, int32_t* idx) {
  return timed_launch(h, GL_TIME_BUILD, "knn launch", [&](hipEvent_t e0, hipEvent_t e1) {
    return gl::launch_knn(x, keys ? keys : x, B, N, C, M, k, dil, dt == GL_BF16, idx, h->sb, e0,
                          e1);
  });
}

// Order the build stream after the update stream's work so far.
gl_status fork_build(gl_lookahead_t h) {
  hipError_t e;
  if ((e = hipEventRecord(h->ev_ready, h->su)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  if ((e = hipStreamWaitEvent(h->sb, h->ev_ready, 0)) != hipSuccess)
    return hip_fail(e, "hipStreamWaitEvent");
  return GL_OK;
}

gl_status mark_built(gl_lookahead_t h) {
  hipError_t e = hipEventRecord(h->ev_built, h->sb);
  if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
  h->pending = true;
  return GL_OK;
}

gl_status join_build(gl_lookahead_t h) {
  if (!h->pending) return GL_OK;
  hipError_t e = hipStreamWaitEvent(h->su, h->ev_built, 0);
  if (e != hipSuccess) return hip_fail(e, "hipStreamWaitEvent");
  h->pending = false;
  return GL_OK;
}

struct BlockArgs {
  const void* x_in;
  int B, H, W, C, pool_r;
  void* keys_ws;
  const int32_t* idx_use;
  int k;
  const void* Wt;
  const void* bias;
  gl_dtype dt;
  void* x_out;
  int32_t* idx_next;
  int dil_next;
  void* ws;          // MRConv workspace (two-pass form), caller-owned
  size_t ws_bytes;
};

gl_status check_block(const BlockArgs& a, int* rt) {
  const int N = a.H * a.W;
  const bool pooled = a.pool_r > 1;
  const int M = pooled ? (a.H / a.pool_r) * (a.W / a.pool_r) : N;
  gl_status s;
  if (a.H < 1 || a.W < 1 || a.pool_r < 1)
    return fail(GL_ERR_BAD_SHAPE, "block: bad grid H=%d W=%d r=%d", a.H, a.W, a.pool_r);
  if (pooled) {
    if (!a.keys_ws) return fail(GL_ERR_NULL_PTR, "block: pool_r > 1 needs keys_ws");
    if ((s = check_pool(a.x_in, a.B, a.H, a.W, a.C, a.pool_r, a.dt, a.keys_ws)) != GL_OK) return s;
  }
  const void* keys = pooled ? a.keys_ws : nullptr;
  if ((s = check_mrconv(a.x_in, a.B, N, a.C, keys, M, a.idx_use, a.k, a.Wt, a.bias, a.C, a.dt,
                        a.x_out, rt)) != GL_OK)
    return s;
  if (pooled && overlap(a.x_out, (size_t)a.B * N * a.C * esize(a.dt), a.keys_ws,
                        (size_t)a.B * M * a.C * esize(a.dt)))
    return fail(GL_ERR_ALIAS, "block: x_out overlaps keys_ws");
  if (a.idx_next) {
    if ((s = check_knn(a.x_in, a.B, N, a.C, keys, M, a.k, a.dil_next, a.dt, a.idx_next)) != GL_OK)
      return s;
    const size_t ib = (size_t)a.B * N * a.k * 4;
    if (overlap(a.idx_next, ib, a.idx_use, ib))
      return fail(GL_ERR_ALIAS, "block: idx_next overlaps idx_use");
    if (overlap(a.idx_next, ib, a.x_out, (size_t)a.B * N * a.C * esize(a.dt)))
      return fail(GL_ERR_ALIAS, "block: idx_next overlaps x_out");
  }
  const size_t xb = (size_t)a.B * N * a.C * esize(a.dt), ib = (size_t)a.B * N * a.k * 4;
  return check_ws("block", mrconv_ws_need(a.B, N, a.C, a.k, a.C, a.dt, *rt), a.ws, a.ws_bytes,
                  {{a.x_in, xb}, {a.x_out, xb}, {a.idx_use, ib}, {a.idx_next, a.idx_next ? ib : 0},
                   {a.keys_ws, pooled ? (size_t)a.B * M * a.C * esize(a.dt) : 0}});
}

// Enqueue one lookahead block whose arguments were checked.
gl_status enqueue_block(gl_lookahead_t h, const BlockArgs& a, int rt, bool do_pool) {
  const int N = a.H * a.W;
  const bool pooled = a.pool_r > 1;
  const int M = pooled ? (a.H / a.pool_r) * (a.W / a.pool_r) : N;
  const void* keys = pooled ? a.keys_ws : a.x_in;
  gl_status s;
  hipError_t e;
  if ((s = join_build(h)) != GL_OK) return s;  // idx_use is ready; old buffers are free
  if (pooled && do_pool) {
    e = gl::launch_pool(a.x_in, a.keys_ws, a.B, a.H, a.W, a.C, a.pool_r, a.dt == GL_BF16, h->su);
    if (e != hipSuccess) return hip_fail(e, "pool launch");
  }
  if (a.idx_next) {
    if ((s = fork_build(h)) != GL_OK) return s;
    if ((s = enqueue_build(h, a.x_in, a.B, N, a.C, pooled ? a.keys_ws : nullptr, M, a.k,
                           a.dil_next, a.dt, a.idx_next)) != GL_OK)
      return s;
    if ((s = mark_built(h)) != GL_OK) return s;
  }
  void* ws = block_ws(a.B, N, a.C, a.k, a.dt, rt, a.ws);
  return timed_launch(h, GL_TIME_UPDATE, "mrconv launch", [&](hipEvent_t e0, hipEvent_t e1) {
    return gl::launch_mrconv(a.x_in, keys, a.idx_use, a.Wt, a.bias, a.x_out, a.B, N, M, a.C, a.C,
                             a.k, a.dt == GL_BF16, rt, ws, h->su, e0, e1);
  });
}

}  // namespace

extern "C" {

int gl_version(void) { return GL_VERSION; }

const char* gl_status_string(gl_status s) {
  switch (s) {
    case GL_OK: return "GL_OK";
    case GL_ERR_NULL_PTR: return "GL_ERR_NULL_PTR";
    case GL_ERR_BAD_SHAPE: return "GL_ERR_BAD_SHAPE";
    case GL_ERR_BAD_K: return "GL_ERR_BAD_K";
    case GL_ERR_UNSUPPORTED: return "GL_ERR_UNSUPPORTED";
    case GL_ERR_ALIGNMENT: return "GL_ERR_ALIGNMENT";
    case GL_ERR_ALIAS: return "GL_ERR_ALIAS";
    case GL_ERR_HIP: return "GL_ERR_HIP";
    case GL_ERR_BAD_HANDLE: return "GL_ERR_BAD_HANDLE";
    case GL_ERR_WORKSPACE: return "GL_ERR_WORKSPACE";
  }
  return "GL_ERR_UNKNOWN";
}

const char* gl_last_error(void) { return g_last_error.c_str(); }

gl_status gl_knn_graph(const void* x, int B, int N, int C, const void* keys, int M, int k,
                       int dilation, gl_dtype dt, int32_t* idx_out, hipStream_t stream) {
  gl_status s = check_knn(x, B, N, C, keys, M, k, dilation, dt, idx_out);
  if (s != GL_OK) return s;
  hipError_t e = gl::launch_knn(x, keys ? keys : x, B, N, C, M, k, dilation, dt == GL_BF16,
                                idx_out, stream);
  return e == hipSuccess ? GL_OK : hip_fail(e, "knn launch");
}

gl_status gl_pool_keys(const void* x, int B, int H, int W, int C, int r, gl_dtype dt,
                       void* keys_out, hipStream_t stream) {
  gl_status s = check_pool(x, B, H, W, C, r, dt, keys_out);
  if (s != GL_OK) return s;
  hipError_t e = gl::launch_pool(x, keys_out, B, H, W, C, r, dt == GL_BF16, stream);
  return e == hipSuccess ? GL_OK : hip_fail(e, "pool launch");
}

gl_status gl_max_pool_nodes(const void* x, int B, int H, int W, int C, int r, gl_dtype dt,
                            void* out, hipStream_t stream) {
  gl_status s = check_pool(x, B, H, W, C, r, dt, out);
  if (s != GL_OK) return s;
  hipError_t e = gl::launch_pool(x, out, B, H, W, C, r, dt == GL_BF16, stream, true);
  return e == hipSuccess ? GL_OK : hip_fail(e, "max pool launch");
}

namespace {

size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

// Workspace of gl_mrconv_heads: none for the per-head kernel; else the dense
// block-diagonal W expanded from Wh (then the two-pass rows when the fused
// tile does not fit LDS).
size_t heads_ws_need(int B, int N, int C, int k, int heads, gl_dtype dt, int rt) {
  if (heads == 1) return mrconv_ws_need(B, N, C, k, C, dt, rt);  // Wh is the dense W
  if (rt > 0 && gl::mrconv_headw_steps(C / heads, dt == GL_BF16)) return 0;
  return align256((size_t)C * 2 * C * esize(dt)) + (rt > 0 ? 0 : mrconv_ws_need(B, N, C, k, C, dt, rt));
}

}  // namespace

size_t gl_mrconv_heads_workspace_bytes(int B, int N, int C, int k, int heads, gl_dtype dt) {
  if (B < 1 || N < 1 || C < 1 || k < 1 || k > GL_MAX_K || !dtype_ok(dt) || !size_ok(B, N, C) ||
      heads < 1 || C % heads)
    return 0;
  return heads_ws_need(B, N, C, k, heads, dt, mrconv_rt(C, k, dt));
}

size_t gl_mrconv_workspace_bytes(int B, int N, int C, int k, int Cout, gl_dtype dt) {
  if (B < 1 || N < 1 || C < 1 || Cout < 1 || k < 1 || k > GL_MAX_K || !dtype_ok(dt) ||
      !size_ok(B, N, C))
    return 0;
  return mrconv_ws_need(B, N, C, k, Cout, dt, mrconv_rt(C, k, dt));
}

namespace {

// Checks of gl_mrconv / gl_mrconv_heads and of the caller's workspace.
gl_status check_mrconv_call(const char* who, const void* x, int B, int N, int C, const void* keys,
                            int M, const int32_t* idx, int k, const void* W, const void* bias,
                            int Cout, gl_dtype dt, const void* out, const void* ws,
                            size_t ws_bytes, int* rt) {
  gl_status s = check_mrconv(x, B, N, C, keys, M, idx, k, W, bias, Cout, dt, out, rt);
  if (s != GL_OK) return s;
  const size_t es = esize(dt);
  return check_ws(who, mrconv_ws_need(B, N, C, k, Cout, dt, *rt), ws, ws_bytes,
                  {{x, (size_t)B * N * C * es}, {keys, keys ? (size_t)B * M * C * es : 0},
                   {idx, (size_t)B * N * k * 4}, {W, (size_t)Cout * 2 * C * es},
                   {bias, bias ? (size_t)Cout * es : 0}, {out, (size_t)B * N * Cout * es}});
}

}  // namespace

gl_status gl_mrconv(const void* x, int B, int N, int C, const void* keys, int M,
                    const int32_t* idx, int k, const void* W, const void* bias, int Cout,
                    gl_dtype dt, void* out, void* workspace, size_t workspace_bytes,
                    hipStream_t stream) {
  int rt = 0;
  gl_status s = check_mrconv_call("mrconv", x, B, N, C, keys, M, idx, k, W, bias, Cout, dt, out,
                                  workspace, workspace_bytes, &rt);
  if (s != GL_OK) return s;
  hipError_t e = gl::launch_mrconv(x, keys ? keys : x, idx, W, bias, out, B, N, M, C, Cout, k,
                                   dt == GL_BF16, rt, workspace, stream);
  return e == hipSuccess ? GL_OK : hip_fail(e, "mrconv launch");
}

gl_status gl_mrconv_heads(const void* x, int B, int N, int C, const void* keys, int M,
                          const int32_t* idx, int k, const void* Wh, const void* bias, int heads,
                          gl_dtype dt, void* out, void* workspace, size_t workspace_bytes,
                          hipStream_t stream) {
  if (heads < 1 || C < 1 || C % heads)
    return fail(GL_ERR_BAD_SHAPE, "mrconv_heads: heads=%d must divide C=%d", heads, C);
  const int hd = C / heads;
  const size_t es = esize(dt);
  const size_t whb = (size_t)C * 2 * hd * es;
  int rt = 0;
  gl_status s = check_mrconv(x, B, N, C, keys, M, idx, k, Wh, bias, C, dt, out, &rt, whb);
  if (s != GL_OK) return s;
  s = check_ws("mrconv_heads", heads_ws_need(B, N, C, k, heads, dt, rt), workspace,
               workspace_bytes,
               {{x, (size_t)B * N * C * es}, {keys, keys ? (size_t)B * M * C * es : 0},
                {idx, (size_t)B * N * k * 4}, {Wh, whb}, {bias, bias ? (size_t)C * es : 0},
                {out, (size_t)B * N * C * es}});
  if (s != GL_OK) return s;
  const int dtb = dt == GL_BF16;
  gl::MrArgs a = gl::make_mr_args(x, keys ? keys : x, idx, Wh, bias, out, B, N, M, C, C, k);
  a.heads = heads;
  hipError_t e;
  if (heads == 1) {
    // one head: Wh [1, C, 2C] is the dense [W_x | W_m]
    a.heads = 1;
    e = gl::launch_mrconv_args(a, dtb, rt, workspace, stream);
  } else if (rt > 0 && gl::mrconv_headw_steps(hd, dtb)) {
    e = gl::launch_mrconv_headw(a, dtb, rt, stream);
  } else {
    // expand Wh into the dense block-diagonal [C, 2C] in the workspace; the
    // fused multi-head tile skips its all-zero steps, the two-pass form (the
    // tile does not fit LDS) runs the dense product
    char* wd = static_cast<char*>(workspace);
    e = gl::launch_expand_heads(Wh, wd, C, heads, dtb, stream);
    if (e == hipSuccess) {
      a.W = wd;
      if (rt < 1) a.heads = 1;
      e = gl::launch_mrconv_args(a, dtb, rt, wd + align256((size_t)C * 2 * C * es), stream);
    }
  }
  return e == hipSuccess ? GL_OK : hip_fail(e, "mrconv_heads launch");
}

gl_status gl_lookahead_create(hipStream_t s_update, hipStream_t s_build, gl_lookahead_t* out) {
  if (!out) return fail(GL_ERR_NULL_PTR, "lookahead_create: out is NULL");
  *out = nullptr;
  gl_lookahead* h = new gl_lookahead();
  h->magic = kHandleMagic;
  h->su = s_update;
  h->sb = s_build;
  h->pending = false;
  h->prof_max = 0;
  h->prof_n[0] = h->prof_n[1] = h->prof_n[2] = h->prof_n[3] = 0;
  hipError_t e = hipEventCreateWithFlags(&h->ev_ready, hipEventDisableTiming);
  if (e != hipSuccess) {
    delete h;
    return hip_fail(e, "hipEventCreate");
  }
  e = hipEventCreateWithFlags(&h->ev_built, hipEventDisableTiming);
  if (e != hipSuccess) {
    (void)hipEventDestroy(h->ev_ready);
    delete h;
    return hip_fail(e, "hipEventCreate");
  }
  *out = h;
  return GL_OK;
}

gl_status gl_lookahead_destroy(gl_lookahead_t h) {
  if (!handle_ok(h)) return fail(GL_ERR_BAD_HANDLE, "lookahead_destroy: bad handle");
  free_profiling(h);
  (void)hipEventDestroy(h->ev_ready);
  (void)hipEventDestroy(h->ev_built);
  h->magic = 0;
  delete h;
  return GL_OK;
}

gl_status gl_lookahead_set_profiling(gl_lookahead_t h, int max_records) {
  if (!handle_ok(h)) return fail(GL_ERR_BAD_HANDLE, "set_profiling: bad handle");
  if (max_records < 0 || max_records > 1 << 20)
    return fail(GL_ERR_BAD_SHAPE, "set_profiling: max_records=%d", max_records);
  free_profiling(h);
  for (int w = 0; w < 4; ++w) {
    for (int i = 0; i < max_records; ++i) {
      hipEvent_t a, b;
      hipError_t e = hipEventCreate(&a);
      if (e != hipSuccess) {
        free_profiling(h);
        return hip_fail(e, "hipEventCreate");
      }
      if ((e = hipEventCreate(&b)) != hipSuccess) {
        (void)hipEventDestroy(a);
        free_profiling(h);
        return hip_fail(e, "hipEventCreate");
      }
      h->prof[w].emplace_back(a, b);
    }
  }
  h->prof_max = max_records;
  return GL_OK;
}

gl_status gl_lookahead_kernel_times(gl_lookahead_t h, int which, float* ms_out, int cap,
                                    int* n_out) {
  if (!handle_ok(h)) return fail(GL_ERR_BAD_HANDLE, "kernel_times: bad handle");
  if (which < GL_TIME_BUILD || which > GL_TIME_LINEAR)
    return fail(GL_ERR_UNSUPPORTED, "kernel_times: which=%d", which);
  if (!n_out || (cap > 0 && !ms_out)) return fail(GL_ERR_NULL_PTR, "kernel_times: null output");
  const int n = h->prof_n[which] < cap ? h->prof_n[which] : cap;
  for (int i = 0; i < n; ++i) {
    const auto& p = h->prof[which][i];
    hipError_t e = hipEventSynchronize(p.second);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    if ((e = hipEventElapsedTime(&ms_out[i], p.first, p.second)) != hipSuccess)
      return hip_fail(e, "hipEventElapsedTime");
  }
  *n_out = n;
  h->prof_n[which] = 0;
  return GL_OK;
}

gl_status gl_lookahead_bootstrap(gl_lookahead_t h, const void* x0, int B, int H, int W, int C,
                                 int pool_r, void* keys_ws, int k, int dilation0, gl_dtype dt,
                                 int32_t* idx0) {
  if (!handle_ok(h)) return fail(GL_ERR_BAD_HANDLE, "bootstrap: bad handle");
  if (H < 1 || W < 1 || pool_r < 1) return fail(GL_ERR_BAD_SHAPE, "bootstrap: bad grid");
  const bool pooled = pool_r > 1;
  const int N = H * W, M = pooled ? (H / pool_r) * (W / pool_r) : N;
  gl_status s;
  if (pooled) {
    if (!keys_ws) return fail(GL_ERR_NULL_PTR, "bootstrap: pool_r > 1 needs keys_ws");
    if ((s = check_pool(x0, B, H, W, C, pool_r, dt, keys_ws)) != GL_OK) return s;
  }
  if ((s = check_knn(x0, B, N, C, pooled ? keys_ws : nullptr, M, k, dilation0, dt, idx0)) != GL_OK)
    return s;
  if ((s = join_build(h)) != GL_OK) return s;
  if (pooled) {
    hipError_t e = gl::launch_pool(x0, keys_ws, B, H, W, C, pool_r, dt == GL_BF16, h->su);
    if (e != hipSuccess) return hip_fail(e, "pool launch");
  }
  if ((s = fork_build(h)) != GL_OK) return s;
  if ((s = enqueue_build(h, x0, B, N, C, pooled ? keys_ws : nullptr, M, k, dilation0, dt, idx0)) !=
      GL_OK)
    return s;
  return mark_built(h);
}

size_t gl_graphleap_workspace_bytes(int B, int H, int W, int C, int pool_r, int k, gl_dtype dt) {
  if (H < 1 || W < 1 || pool_r < 1 || H % pool_r || W % pool_r) return 0;
  return gl_mrconv_workspace_bytes(B, H * W, C, k, C, dt);
}

gl_status gl_graphleap_block(gl_lookahead_t h, const void* x_in, int B, int H, int W, int C,
                             int pool_r, void* keys_ws, const int32_t* idx_use, int k,
                             const void* Wt, const void* bias, gl_dtype dt, void* x_out,
                             int32_t* idx_next, int dilation_next, void* workspace,
                             size_t workspace_bytes) {
  if (!handle_ok(h)) return fail(GL_ERR_BAD_HANDLE, "graphleap_block: bad handle");
  BlockArgs a{x_in, B, H, W, C, pool_r, keys_ws, idx_use, k, Wt, bias, dt, x_out, idx_next,
              dilation_next, workspace, workspace_bytes};
  int rt = 0;
  gl_status s = check_block(a, &rt);
  if (s != GL_OK) return s;
  return enqueue_block(h, a, rt, true);
}

gl_status gl_graphleap_stack(gl_lookahead_t h, const void* x0, int B, int H, int W, int C,
                             int pool_r, int L, int k, const int* dilations, const void* Ws,
                             const void* bs, gl_dtype dt, gl_schedule schedule, void* x_ws,
                             int32_t* idx_ws, void* keys_ws, void* x_out, void* workspace,
                             size_t workspace_bytes) {
  if (!handle_ok(h)) return fail(GL_ERR_BAD_HANDLE, "graphleap_stack: bad handle");
  if (!x0 || !dilations || !Ws || !x_ws || !idx_ws || !x_out)
    return fail(GL_ERR_NULL_PTR, "graphleap_stack: x0, dilations, Ws, x_ws, idx_ws, x_out required");
  if (schedule != GL_SCHED_LOOKAHEAD && schedule != GL_SCHED_STANDARD &&
      schedule != GL_SCHED_LOOKAHEAD_FUSED)
    return fail(GL_ERR_UNSUPPORTED, "graphleap_stack: unknown schedule %d", (int)schedule);
  if (L < 1 || L > 4096) return fail(GL_ERR_BAD_SHAPE, "graphleap_stack: L=%d", L);
  if (!dtype_ok(dt)) return fail(GL_ERR_UNSUPPORTED, "graphleap_stack: unknown dtype");
  if (H < 1 || W < 1 || pool_r < 1 || B < 1 || C < 1 || !size_ok(B, (long long)H * W, C))
    return fail(GL_ERR_BAD_SHAPE, "graphleap_stack: bad shape");
  const int N = H * W;
  const bool pooled = pool_r > 1;
  const size_t es = esize(dt);
  const size_t xbytes = (size_t)B * N * C * es, ibytes = (size_t)B * N * k * 4;
  const size_t wbytes = (size_t)C * 2 * C * es, bbytes = (size_t)C * es;
  const int M = pooled ? (H / pool_r) * (W / pool_r) : N;
  const size_t kbytes = pooled ? (size_t)B * M * C * es : 0;
  if (overlap(x_out, xbytes, x_ws, 2 * xbytes) || overlap(x_out, xbytes, idx_ws, 2 * ibytes) ||
      overlap(x_out, xbytes, keys_ws, kbytes) || overlap(x_out, xbytes, x0, xbytes) ||
      overlap(x_ws, 2 * xbytes, idx_ws, 2 * ibytes) || overlap(x_ws, 2 * xbytes, keys_ws, kbytes) ||
      overlap(x_ws, 2 * xbytes, x0, xbytes) || overlap(idx_ws, 2 * ibytes, keys_ws, kbytes) ||
      overlap(idx_ws, 2 * ibytes, x0, xbytes) || overlap(keys_ws, kbytes, x0, xbytes))
    return fail(GL_ERR_ALIAS, "graphleap_stack: workspaces overlap each other or x0");
  if (overlap(workspace, workspace_bytes, x_out, xbytes) ||
      overlap(workspace, workspace_bytes, x_ws, 2 * xbytes) ||
      overlap(workspace, workspace_bytes, idx_ws, 2 * ibytes) ||
      overlap(workspace, workspace_bytes, keys_ws, kbytes) ||
      overlap(workspace, workspace_bytes, x0, xbytes))
    return fail(GL_ERR_ALIAS, "graphleap_stack: workspace overlaps another buffer");
  char* xw[2] = {static_cast<char*>(x_ws), static_cast<char*>(x_ws) + xbytes};
  int32_t* iw[2] = {idx_ws, idx_ws + (size_t)B * N * k};
  const char* Wb = static_cast<const char*>(Ws);
  const char* bb = static_cast<const char*>(bs);

  // check every block before enqueuing anything
  std::vector<BlockArgs> blocks(L);
  std::vector<int> rts(L);
  for (int l = 0; l < L; ++l) {
    BlockArgs& a = blocks[l];
    a = BlockArgs{l == 0 ? x0 : xw[(l - 1) & 1], B, H, W, C, pool_r, keys_ws, iw[0], k,
                  Wb + l * wbytes, bb ? bb + l * bbytes : nullptr, dt,
                  l == L - 1 ? x_out : static_cast<void*>(xw[l & 1]), nullptr, 1, workspace,
                  workspace_bytes};
    if (schedule != GL_SCHED_STANDARD && l + 1 < L) {
      a.idx_next = iw[1];
      a.dil_next = dilations[l + 1];
    }
    gl_status s = check_block(a, &rts[l]);
    if (s != GL_OK) return s;
    if ((s = check_knn(a.x_in, B, N, C, pooled ? keys_ws : nullptr, M, k, dilations[l], dt, iw[0])) !=
        GL_OK)
      return s;
  }

  gl_status s;
  if (schedule == GL_SCHED_STANDARD) {
    if ((s = join_build(h)) != GL_OK) return s;
    for (int l = 0; l < L; ++l) {
      BlockArgs a = blocks[l];
      hipError_t e;
      if (pooled) {
        e = gl::launch_pool(a.x_in, keys_ws, B, H, W, C, pool_r, dt == GL_BF16, h->su);
        if (e != hipSuccess) return hip_fail(e, "pool launch");
      }
      e = gl::launch_knn(a.x_in, pooled ? keys_ws : a.x_in, B, N, C, M, k, dilations[l],
                         dt == GL_BF16, iw[0], h->su);
      if (e != hipSuccess) return hip_fail(e, "knn launch");
      void* ws = block_ws(B, N, C, k, dt, rts[l], workspace);
      e = gl::launch_mrconv(a.x_in, pooled ? keys_ws : a.x_in, iw[0], a.Wt, a.bias, a.x_out, B, N,
                            M, C, C, k, dt == GL_BF16, rts[l], ws, h->su);
      if (e != hipSuccess) return hip_fail(e, "mrconv launch");
    }
    return GL_OK;
  }

  if (schedule == GL_SCHED_LOOKAHEAD_FUSED) {
    // everything on the update stream; each block is one launch holding the
    // build tiles of the next graph and the update tiles of this block
    if ((s = join_build(h)) != GL_OK) return s;
    hipError_t e;
    const int dtb = dt == GL_BF16;
    const void* keys0 = pooled ? keys_ws : x0;
    if (pooled && (e = gl::launch_pool(x0, keys_ws, B, H, W, C, pool_r, dtb, h->su)) != hipSuccess)
      return hip_fail(e, "pool launch");
    if ((s = timed_launch(h, GL_TIME_BUILD, "knn launch", [&](hipEvent_t e0, hipEvent_t e1) {
           return gl::launch_knn(x0, keys0, B, N, C, M, k, dilations[0], dtb, iw[0], h->su, e0, e1);
         })) != GL_OK)
      return s;
    int cur = 0;
    for (int l = 0; l < L; ++l) {
      const BlockArgs& a = blocks[l];
      const void* keys = pooled ? keys_ws : a.x_in;
      if (l > 0 && pooled &&
          (e = gl::launch_pool(a.x_in, keys_ws, B, H, W, C, pool_r, dtb, h->su)) != hipSuccess)
        return hip_fail(e, "pool launch");
      int next = cur;
      const bool build = l + 1 < L && !(l == 0 && dilations[1] == dilations[0]);
      const gl::MrArgs ma = gl::make_mr_args(a.x_in, keys, iw[cur], a.Wt, a.bias, a.x_out, B, N, M,
                                             C, C, k);
      void* ws = block_ws(B, N, C, k, dt, rts[l], workspace);
      if (build && !gl::knn_separate(M, C, dtb) && !ws) {
        next = 1 - cur;
        const gl::KnnArgs ka = gl::make_knn_args(a.x_in, keys, B, N, C, M, k, dilations[l + 1],
                                                 iw[next]);
        s = timed_launch(h, GL_TIME_FUSED, "block launch", [&](hipEvent_t e0, hipEvent_t e1) {
          return gl::launch_block(ka, ma, dtb, rts[l], h->su, e0, e1);
        });
      } else if (build && ws && gl::block_hosts_build(B, N, M, C, B * N, dtb)) {
        // two-pass update (wide W): the build tiles and the gather tiles in one
        // launch, then the GEMM pass; timed together as the block
        next = 1 - cur;
        const gl::KnnArgs ka = gl::make_knn_args(a.x_in, keys, B, N, C, M, k, dilations[l + 1],
                                                 iw[next]);
        s = timed_launch(h, GL_TIME_FUSED, "block launch", [&](hipEvent_t e0, hipEvent_t e1) {
          hipError_t e = gl::launch_block_gather(ka, ma, ws, h->su, e0);
          return e != hipSuccess ? e : gl::launch_mrconv_gemm(ma, dtb, ws, h->su, nullptr, e1);
        });
      } else if (build) {
        // large key sets: the build kernel, then the update, in stream order
        next = 1 - cur;
        s = timed_launch(h, GL_TIME_BUILD, "knn launch", [&](hipEvent_t e0, hipEvent_t e1) {
          return gl::launch_knn(a.x_in, keys, B, N, C, M, k, dilations[l + 1], dtb, iw[next], h->su,
                                e0, e1);
        });
        if (s != GL_OK) return s;
        s = timed_launch(h, GL_TIME_UPDATE, "mrconv launch", [&](hipEvent_t e0, hipEvent_t e1) {
          return gl::launch_mrconv(a.x_in, keys, iw[cur], a.Wt, a.bias, a.x_out, B, N, M, C, C, k,
                                   dtb, rts[l], ws, h->su, e0, e1);
        });
      } else {
        s = timed_launch(h, GL_TIME_UPDATE, "mrconv launch", [&](hipEvent_t e0, hipEvent_t e1) {
          return gl::launch_mrconv(a.x_in, keys, iw[cur], a.Wt, a.bias, a.x_out, B, N, M, C, C, k,
                                   dtb, rts[l], ws, h->su, e0, e1);
        });
      }
      if (s != GL_OK) return s;
      cur = next;
    }
    return GL_OK;
  }

  // lookahead: Ghat^0 = G(X^0, d_0) into iw[0]
  if ((s = gl_lookahead_bootstrap(h, x0, B, H, W, C, pool_r, keys_ws, k, dilations[0], dt, iw[0])) !=
      GL_OK)
    return s;
  int cur = 0;  // buffer holding Ghat^l
  for (int l = 0; l < L; ++l) {
    BlockArgs a = blocks[l];
    a.idx_use = iw[cur];
    int next = cur;
    a.idx_next = nullptr;
    if (l + 1 < L) {
      if (l == 0 && dilations[1] == dilations[0]) {
        next = cur;  // Ghat^1 = G(X^0, d_1) is the bootstrap graph itself
      } else {
        next = 1 - cur;
        a.idx_next = iw[next];
        a.dil_next = dilations[l + 1];
      }
    }
    if ((s = enqueue_block(h, a, rts[l], /*do_pool=*/l > 0)) != GL_OK) return s;
    cur = next;
  }
  return GL_OK;
}

}  // extern "C"

// ===========================================================================
// The full ViG block (Sec. III Eq. 11-15, Alg. 1)
// ===========================================================================
namespace {

gl_status check_linear(const void* x, int R, int K, const void* W, const void* bias, int Cout,
                       gl_act act_in, gl_act act_out, const void* residual, gl_dtype dt,
                       const void* out) {
  if (!x || !W || !out) return fail(GL_ERR_NULL_PTR, "linear: x, W and out are required");
  if (!dtype_ok(dt)) return fail(GL_ERR_UNSUPPORTED, "linear: unknown dtype %d", (int)dt);
  if ((act_in != GL_ACT_NONE && act_in != GL_ACT_GELU) ||
      (act_out != GL_ACT_NONE && act_out != GL_ACT_GELU))
    return fail(GL_ERR_UNSUPPORTED, "linear: unknown activation");
  if (R < 1 || K < 1 || Cout < 1 || !size_ok(R, 1, K) || !size_ok(R, 1, Cout) ||
      !size_ok(Cout, 1, K))
    return fail(GL_ERR_BAD_SHAPE, "linear: bad shape R=%d K=%d Cout=%d", R, K, Cout);
  if (K % vec_width(dt))
    return fail(GL_ERR_UNSUPPORTED, "linear: K=%d must be a multiple of %d", K, vec_width(dt));
  const size_t es = esize(dt);
  if (!aligned(x, 16) || !aligned(W, 16) || !aligned(out, es) || (bias && !aligned(bias, es)) ||
      (residual && !aligned(residual, es)))
    return fail(GL_ERR_ALIGNMENT, "linear: x and W need 16-byte alignment");
  const size_t ob = (size_t)R * Cout * es;
  if (overlap(out, ob, x, (size_t)R * K * es) || overlap(out, ob, W, (size_t)Cout * K * es) ||
      overlap(out, ob, bias, bias ? (size_t)Cout * es : 0) ||
      (residual && residual != out && overlap(out, ob, residual, ob)))
    return fail(GL_ERR_ALIAS, "linear: out overlaps an input");
  return GL_OK;
}

hipError_t run_linear(const void* x, int R, int K, const void* W, const void* bias, int Cout,
                      int act_in, int act_out, const void* residual, gl_dtype dt, void* out,
                      hipStream_t stream, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr) {
  gl::GemmArgs a;
  a.A = x;
  a.W = W;
  a.bias = bias;
  a.residual = residual;
  a.out = out;
  a.R = R;
  a.K = K;
  a.Cout = Cout;
  a.act_in = act_in;
  a.act_out = act_out;
  return gl::launch_gemm_nt(a, dt == GL_BF16, stream, e0, e1);
}

size_t round256(size_t v) { return (v + 255) & ~size_t(255); }

// Workspace carve-up: sigma(Ut) (MRConv's output), Y, FFN hidden H (block and
// stack), the pooled keys of U (pyramid stages), then U, two feature buffers
// and two graphs (stack only).
struct VigWs {
  char* ut;
  char* y;
  char* hid;
  char* u;
  char* x[2];
  char* keys;
  int32_t* idx[2];
  size_t bytes;
};

size_t vig_ws_bytes(int B, int N, int C, int k, gl_dtype dt) {
  const size_t fb = round256((size_t)B * N * C * esize(dt));
  return 10 * fb + 2 * round256((size_t)B * N * k * 4);
}

VigWs vig_ws(void* base, int B, int N, int C, int k, gl_dtype dt) {
  const size_t fb = round256((size_t)B * N * C * esize(dt));
  const size_t ib = round256((size_t)B * N * k * 4);
  char* p = static_cast<char*>(base);
  VigWs w;
  w.ut = p;
  w.y = p + fb;
  w.hid = p + 2 * fb;     // 4 feature buffers: [B, N, 4C]
  w.u = p + 6 * fb;
  w.x[0] = p + 7 * fb;
  w.x[1] = p + 8 * fb;
  w.keys = p + 9 * fb;    // [B, M, C], M <= N
  w.idx[0] = reinterpret_cast<int32_t*>(p + 10 * fb);
  w.idx[1] = reinterpret_cast<int32_t*>(p + 10 * fb + ib);
  w.bytes = vig_ws_bytes(B, N, C, k, dt);
  return w;
}

// The node grid of a full block: N = H*W queries; with r > 1 the graph and
// MRConv use the M = (H/r)*(W/r) keys pooled from U, else M = N and keys = U.
struct VigGrid {
  int B, H, W, C, r;
  int N() const { return H * W; }
  int M() const { return r > 1 ? (H / r) * (W / r) : H * W; }
  bool pooled() const { return r > 1; }
};

bool grid_ok(const VigGrid& g, int k, gl_dtype dt) {
  return g.B >= 1 && g.H >= 1 && g.W >= 1 && g.C >= 1 && g.r >= 1 && k >= 1 && dtype_ok(dt) &&
         g.H % g.r == 0 && g.W % g.r == 0 && size_ok(g.B, (long long)g.H * g.W, g.C);
}

gl_status check_grid(const char* who, const VigGrid& g, int k, gl_dtype dt) {
  if (!grid_ok(g, k, dt))
    return fail(GL_ERR_BAD_SHAPE, "%s: bad shape B=%d H=%d W=%d C=%d pool_r=%d k=%d", who, g.B,
                g.H, g.W, g.C, g.r, k);
  return GL_OK;
}

gl_status check_vig_params(const gl_vig_params* p, int C, gl_dtype dt) {
  if (!p) return fail(GL_ERR_NULL_PTR, "vig: params is NULL");
  if (!p->W_in || !p->W_upd || !p->W_out || !p->W_1 || !p->W_2)
    return fail(GL_ERR_NULL_PTR, "vig: every weight matrix is required");
  const size_t es = esize(dt);
  const void* mats[5] = {p->W_in, p->W_upd, p->W_out, p->W_1, p->W_2};
  const void* bs[5] = {p->b_in, p->b_upd, p->b_out, p->b_1, p->b_2};
  for (int i = 0; i < 5; ++i) {
    if (!aligned(mats[i], 16) || (bs[i] && !aligned(bs[i], es)))
      return fail(GL_ERR_ALIGNMENT, "vig: weights need 16-byte alignment");
  }
  (void)C;
  return GL_OK;
}

// One full block on the handle's streams.  u holds U^l (computed here, and
// pooled into w.keys at pyramid stages, unless u_ready); idx_next (if any)
// receives G(U^l, dil_next).
gl_status enqueue_vig_block(gl_lookahead_t h, const void* x_in, const VigGrid& g, int k,
                            const int32_t* idx_use, const gl_vig_params& p, gl_dtype dt,
                            const VigWs& w, void* u, bool u_ready, int32_t* idx_next,
                            int dil_next, gl_schedule schedule, int rt, void* x_out) {
  const int B = g.B, N = g.N(), M = g.M(), C = g.C, R = B * N, dtb = dt == GL_BF16;
  const void* keys = g.pooled() ? static_cast<const void*>(w.keys) : u;
  gl_status s;
  auto lin = [&](const char* what, const void* xi, int K, const void* W, const void* b, int Co,
                 int ai, int ao, const void* res, void* o) {
    return timed_launch(h, GL_TIME_LINEAR, what, [&](hipEvent_t e0, hipEvent_t e1) {
      return run_linear(xi, R, K, W, b, Co, ai, ao, res, dt, o, h->su, e0, e1);
    });
  };
  if (schedule == GL_SCHED_LOOKAHEAD && (s = join_build(h)) != GL_OK) return s;
  if (!u_ready) {
    if ((s = lin("linear launch (FC1)", x_in, C, p.W_in, p.b_in, C, 0, 0, nullptr, u)) != GL_OK)
      return s;
    if (g.pooled()) {
      hipError_t e = gl::launch_pool(u, w.keys, B, g.H, g.W, C, g.r, dtb, h->su);
      if (e != hipSuccess) return hip_fail(e, "pool launch");
    }
  }
  // the two-pass MRConv's [x | m] rows go to the FFN's hidden-row region,
  // which is free until FFN1 (later on the same stream) overwrites it
  void* mws = block_ws(B, N, C, k, dt, rt, w.hid);
  const bool fused = schedule == GL_SCHED_LOOKAHEAD_FUSED && idx_next &&
                     !gl::knn_separate(M, C, dtb) && !mws;
  // MRConv writes sigma(U~) (GELU before its one rounding): FC2 is its only
  // reader, so the GELU is paid once per element instead of once per FC2
  // output-column tile
  gl::MrArgs ma = gl::make_mr_args(u, keys, idx_use, p.W_upd, p.b_upd, w.ut, B, N, M, C, C, k);
  ma.act_out = 1;
  if (fused) {
    const gl::KnnArgs ka = gl::make_knn_args(u, keys, B, N, C, M, k, dil_next, idx_next);
    s = timed_launch(h, GL_TIME_FUSED, "block launch", [&](hipEvent_t e0, hipEvent_t e1) {
      return gl::launch_block(ka, ma, dtb, rt, h->su, e0, e1);
    });
    if (s != GL_OK) return s;
  } else if (schedule == GL_SCHED_LOOKAHEAD_FUSED && idx_next && mws &&
             gl::block_hosts_build(B, N, M, C, R, dtb)) {
    // two-pass update: the build tiles and the gather tiles in one launch, then
    // the GEMM pass (with the GELU); timed together as the block
    const gl::KnnArgs ka = gl::make_knn_args(u, keys, B, N, C, M, k, dil_next, idx_next);
    s = timed_launch(h, GL_TIME_FUSED, "block launch", [&](hipEvent_t e0, hipEvent_t e1) {
      hipError_t e = gl::launch_block_gather(ka, ma, mws, h->su, e0);
      return e != hipSuccess ? e : gl::launch_mrconv_gemm(ma, dtb, mws, h->su, nullptr, e1);
    });
    if (s != GL_OK) return s;
  } else {
    if (idx_next) {
      if (schedule == GL_SCHED_LOOKAHEAD) {
        if ((s = fork_build(h)) != GL_OK) return s;
        if ((s = enqueue_build(h, u, B, N, C, g.pooled() ? w.keys : nullptr, M, k, dil_next, dt,
                               idx_next)) != GL_OK)
          return s;
        if ((s = mark_built(h)) != GL_OK) return s;
      } else {
        s = timed_launch(h, GL_TIME_BUILD, "knn launch", [&](hipEvent_t e0, hipEvent_t e1) {
          return gl::launch_knn(u, keys, B, N, C, M, k, dil_next, dtb, idx_next, h->su, e0, e1);
        });
        if (s != GL_OK) return s;
      }
    }
    s = timed_launch(h, GL_TIME_UPDATE, "mrconv launch", [&](hipEvent_t e0, hipEvent_t e1) {
      return gl::launch_mrconv_args(ma, dtb, rt, mws, h->su, e0, e1);
    });
    if (s != GL_OK) return s;
  }
  if ((s = lin("linear launch (FC2)", w.ut, C, p.W_out, p.b_out, C, 0, 0, x_in, w.y)) != GL_OK)
    return s;
  if ((s = lin("linear launch (FFN1)", w.y, C, p.W_1, p.b_1, 4 * C, 0, 1, nullptr, w.hid)) != GL_OK)
    return s;
  return lin("linear launch (FFN2)", w.hid, 4 * C, p.W_2, p.b_2, C, 0, 0, w.y, x_out);
}

}  // namespace

extern "C" {

gl_status gl_linear(const void* x, int R, int K, const void* W, const void* bias, int Cout,
                    gl_act act_in, gl_act act_out, const void* residual, gl_dtype dt,
                    void* out, hipStream_t stream) {
  gl_status s = check_linear(x, R, K, W, bias, Cout, act_in, act_out, residual, dt, out);
  if (s != GL_OK) return s;
  hipError_t e = run_linear(x, R, K, W, bias, Cout, act_in, act_out, residual, dt, out, stream);
  return e == hipSuccess ? GL_OK : hip_fail(e, "linear launch");
}

size_t gl_vig_workspace_bytes(int B, int H, int W, int C, int pool_r, int k, gl_dtype dt) {
  const VigGrid g{B, H, W, C, pool_r};
  return grid_ok(g, k, dt) ? vig_ws_bytes(B, g.N(), C, k, dt) : 0;
}

gl_status gl_vig_block(gl_lookahead_t h, const void* x_in, int B, int H, int W, int C, int pool_r,
                       int k, const int32_t* idx_use, const gl_vig_params* p, gl_dtype dt,
                       void* ws, size_t ws_bytes, void* u_out, int32_t* idx_next,
                       int dilation_next, void* x_out) {
  if (!handle_ok(h)) return fail(GL_ERR_BAD_HANDLE, "vig_block: bad handle");
  const VigGrid g{B, H, W, C, pool_r};
  gl_status s;
  if ((s = check_grid("vig_block", g, k, dt)) != GL_OK) return s;
  if ((s = check_vig_params(p, C, dt)) != GL_OK) return s;
  if (!x_in || !idx_use || !ws || !u_out || !x_out)
    return fail(GL_ERR_NULL_PTR, "vig_block: x_in, idx_use, ws, u_out and x_out are required");
  const int N = g.N(), M = g.M();
  const VigWs w = vig_ws(ws, B, N, C, k, dt);
  if (ws_bytes < w.bytes)
    return fail(GL_ERR_BAD_SHAPE, "vig_block: ws_bytes=%zu < %zu", ws_bytes, w.bytes);
  if (!aligned(x_in, 16) || !aligned(u_out, 16) || !aligned(ws, 256) || !aligned(x_out, 16))
    return fail(GL_ERR_ALIGNMENT, "vig_block: x_in, u_out, x_out need 16 bytes, ws 256");
  const void* keys = g.pooled() ? w.keys : nullptr;
  int rt = 0;
  // shapes of every layer: FC1 [C->C], MRConv [2C->C], FC2 [C->C], FFN [C->4C->C]
  if (g.pooled() && (s = check_pool(u_out, B, H, W, C, pool_r, dt, w.keys)) != GL_OK) return s;
  if ((s = check_mrconv(u_out, B, N, C, keys, M, idx_use, k, p->W_upd, p->b_upd, C, dt, x_out,
                        &rt)) != GL_OK)
    return s;
  if (idx_next && (s = check_knn(u_out, B, N, C, keys, M, k, dilation_next, dt, idx_next)) != GL_OK)
    return s;
  const size_t xb = (size_t)B * N * C * esize(dt), ib = (size_t)B * N * k * 4;
  if (overlap(x_out, xb, x_in, xb) || overlap(x_out, xb, u_out, xb) ||
      overlap(x_out, xb, ws, ws_bytes) || overlap(x_out, xb, idx_use, ib) ||
      overlap(x_out, xb, idx_next, idx_next ? ib : 0) || overlap(u_out, xb, x_in, xb) ||
      overlap(u_out, xb, ws, ws_bytes) || overlap(x_in, xb, ws, ws_bytes) ||
      overlap(idx_use, ib, ws, ws_bytes) || overlap(idx_next, idx_next ? ib : 0, ws, ws_bytes) ||
      overlap(idx_next, idx_next ? ib : 0, idx_use, ib))
    return fail(GL_ERR_ALIAS, "vig_block: buffers overlap");
  return enqueue_vig_block(h, x_in, g, k, idx_use, *p, dt, w, u_out, false, idx_next,
                           dilation_next, GL_SCHED_LOOKAHEAD, rt, x_out);
}

gl_status gl_vig_stack(gl_lookahead_t h, const void* x0, int B, int H, int W, int C, int pool_r,
                       int L, int k, const int* dilations, const gl_vig_params* params,
                       gl_dtype dt, gl_schedule schedule, void* ws, size_t ws_bytes,
                       void* x_out) {
  if (!handle_ok(h)) return fail(GL_ERR_BAD_HANDLE, "vig_stack: bad handle");
  if (!x0 || !dilations || !params || !ws || !x_out)
    return fail(GL_ERR_NULL_PTR, "vig_stack: x0, dilations, params, ws and x_out are required");
  if (L < 1) return fail(GL_ERR_BAD_SHAPE, "vig_stack: L=%d", L);
  if (schedule != GL_SCHED_LOOKAHEAD && schedule != GL_SCHED_STANDARD &&
      schedule != GL_SCHED_LOOKAHEAD_FUSED)
    return fail(GL_ERR_UNSUPPORTED, "vig_stack: schedule=%d", (int)schedule);
  const VigGrid g{B, H, W, C, pool_r};
  gl_status s;
  if ((s = check_grid("vig_stack", g, k, dt)) != GL_OK) return s;
  const int N = g.N(), M = g.M();
  const VigWs w = vig_ws(ws, B, N, C, k, dt);
  if (ws_bytes < w.bytes)
    return fail(GL_ERR_BAD_SHAPE, "vig_stack: ws_bytes=%zu < %zu", ws_bytes, w.bytes);
  if (!aligned(x0, 16) || !aligned(x_out, 16) || !aligned(ws, 256))
    return fail(GL_ERR_ALIGNMENT, "vig_stack: x0, x_out need 16 bytes, ws 256");
  const size_t xb = (size_t)B * N * C * esize(dt);
  if (overlap(x_out, xb, x0, xb) || overlap(x_out, xb, ws, ws_bytes) || overlap(x0, xb, ws, ws_bytes))
    return fail(GL_ERR_ALIAS, "vig_stack: x_out, x0 and ws must not overlap");
  const void* keys = g.pooled() ? static_cast<const void*>(w.keys) : w.u;
  const void* keys_arg = g.pooled() ? w.keys : nullptr;
  int rt = 0;
  if (g.pooled() && (s = check_pool(w.u, B, H, W, C, pool_r, dt, w.keys)) != GL_OK) return s;
  for (int l = 0; l < L; ++l) {
    if ((s = check_vig_params(&params[l], C, dt)) != GL_OK) return s;
    if ((s = check_knn(w.u, B, N, C, keys_arg, M, k, dilations[l], dt, w.idx[0])) != GL_OK) return s;
    if ((s = check_mrconv(w.u, B, N, C, keys_arg, M, w.idx[0], k, params[l].W_upd, params[l].b_upd,
                          C, dt, w.ut, &rt)) != GL_OK)
      return s;
  }
  const int dtb = dt == GL_BF16;
  // U^l = FC1(X^l) into w.u, pooled into w.keys at pyramid stages
  auto project = [&](const void* xi, int l) -> gl_status {
    gl_status st = timed_launch(h, GL_TIME_LINEAR, "linear launch (FC1)",
                                [&](hipEvent_t e0, hipEvent_t e1) {
      return run_linear(xi, B * N, C, params[l].W_in, params[l].b_in, C, 0, 0, nullptr, dt, w.u,
                        h->su, e0, e1);
    });
    if (st != GL_OK || !g.pooled()) return st;
    hipError_t e = gl::launch_pool(w.u, w.keys, B, H, W, C, pool_r, dtb, h->su);
    return e == hipSuccess ? GL_OK : hip_fail(e, "pool launch");
  };
  auto build = [&](int dil, int32_t* idx) {
    return timed_launch(h, GL_TIME_BUILD, "knn launch", [&](hipEvent_t e0, hipEvent_t e1) {
      return gl::launch_knn(w.u, keys, B, N, C, M, k, dil, dtb, idx, h->su, e0, e1);
    });
  };
  if ((s = join_build(h)) != GL_OK) return s;
  if (schedule == GL_SCHED_STANDARD) {
    for (int l = 0; l < L; ++l) {
      const void* xi = l == 0 ? x0 : w.x[(l - 1) & 1];
      void* xo = l == L - 1 ? x_out : w.x[l & 1];
      if ((s = project(xi, l)) != GL_OK) return s;
      if ((s = build(dilations[l], w.idx[0])) != GL_OK) return s;
      if ((s = enqueue_vig_block(h, xi, g, k, w.idx[0], params[l], dt, w, w.u, true, nullptr, 0,
                                 schedule, rt, xo)) != GL_OK)
        return s;
    }
    return GL_OK;
  }
  // lookahead: U^0, then Ghat^0 = G(U^0, d_0)
  if ((s = project(x0, 0)) != GL_OK) return s;
  if ((s = build(dilations[0], w.idx[0])) != GL_OK) return s;
  int cur = 0;
  for (int l = 0; l < L; ++l) {
    const void* xi = l == 0 ? x0 : w.x[(l - 1) & 1];
    void* xo = l == L - 1 ? x_out : w.x[l & 1];
    int next = cur;
    int32_t* idx_next = nullptr;
    if (l + 1 < L && !(l == 0 && dilations[1] == dilations[0])) {
      next = 1 - cur;
      idx_next = w.idx[next];
    }
    if ((s = enqueue_vig_block(h, xi, g, k, w.idx[cur], params[l], dt, w, w.u, l == 0, idx_next,
                               idx_next ? dilations[l + 1] : 0, schedule, rt, xo)) != GL_OK)
      return s;
    cur = next;
  }
  return join_build(h);
}

}  // extern "C"

// ===========================================================================
// MRConv that allocates nothing and takes no workspace (gl_mrconv_noalloc).
// ===========================================================================
namespace {

// The [x | m] rows of the two-pass MRConv of gl_mrconv_noalloc.  Each device
// the library runs on holds its own copy until the process ends.  In host code
// this name stands for a host-side shadow, not device memory: kernels get the
// device address taken with hipGetSymbolAddress (scratch_ptr below).
static __device__ __align__(256) char scratch[GL_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// Device address of `scratch` on the current device, taken once per device
// (with that device current) and kept.  The stream must belong to it.
gl_status scratch_ptr(hipStream_t stream, void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (stream) {
    int sdev = -1;
    if ((e = hipStreamGetDevice(stream, &sdev)) != hipSuccess) return hip_fail(e, "hipStreamGetDevice");
    if (sdev != dev)
      return fail(GL_ERR_UNSUPPORTED, "mrconv_noalloc: the stream is on device %d, the current device is %d",
                  sdev, dev);
  }
  if (dev < 0 || dev >= kMaxDevices)
    return fail(GL_ERR_UNSUPPORTED, "mrconv_noalloc: device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess)
      return hip_fail(e, "hipGetSymbolAddress (scratch)");
    if (!p) return fail(GL_ERR_HIP, "hipGetSymbolAddress (scratch) returned NULL");
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return GL_OK;
}

}  // namespace

extern "C" gl_status gl_mrconv_noalloc(const void* x, int B, int N, int C, const void* keys, int M,
                                       const int32_t* idx, int k, const void* W, const void* bias,
                                       int Cout, gl_dtype dt, void* out, hipStream_t stream) {
  int rt = 0;
  gl_status s = check_mrconv(x, B, N, C, keys, M, idx, k, W, bias, Cout, dt, out, &rt);
  if (s != GL_OK) return s;
  const size_t need = mrconv_ws_need(B, N, C, k, Cout, dt, rt);
  if (need > (size_t)GL_NOALLOC_SCRATCH_BYTES)
    return fail(GL_ERR_WORKSPACE,
                "mrconv_noalloc: this layer needs %zu bytes of scratch, beyond the library's %zu "
                "(use gl_mrconv with a workspace)",
                need, (size_t)GL_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  if (need && (s = scratch_ptr(stream, &ws)) != GL_OK) return s;
  // the gather writes every [x | m] row the GEMM reads: nothing to clear
  hipError_t e = gl::launch_mrconv(x, keys ? keys : x, idx, W, bias, out, B, N, M, C, Cout, k,
                                   dt == GL_BF16, rt, ws, stream);
  return e == hipSuccess ? GL_OK : hip_fail(e, "mrconv launch");
}
