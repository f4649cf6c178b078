#include <algorithm>
// C ABI of the triangle-attention library: argument checks, workspace
// layout and launch sequencing.  Every check runs before the first HIP call.
#include <math.h>
#include <stdint.h>

#include <mutex>
#include <type_traits>

#include "kernels.h"
#include "triattn.h"

namespace {

using triattn::Geom;

constexpr int64_t MAX_N = 8192;
constexpr int64_t MAX_H = 64;

size_t round256(size_t x) { return (x + 255) & ~(size_t)255; }

// d = 32 everywhere; the whole-map and batched calls also take d = 16
// (padded to 32) and d = 64 (the register-staged kernels).
int check_shape(int node, int dtype, int64_t n, int64_t h, int64_t d, bool whole = false) {
  if (node != TRIATTN_STARTING && node != TRIATTN_ENDING) return TRIATTN_ERR_INVALID_ARG;
  if (dtype != TRIATTN_F32 && dtype != TRIATTN_BF16) return TRIATTN_ERR_INVALID_ARG;
  if (n < 1 || n > MAX_N || h < 1 || h > MAX_H || d < 1) return TRIATTN_ERR_INVALID_ARG;
  if (d != triattn::HEAD_DIM && !(whole && (d == 16 || d == 64))) return TRIATTN_ERR_UNSUPPORTED;
  return TRIATTN_OK;
}

// Channels per head the kernels run with: 64 for d = 64, 16 for bf16 d = 16
// (the DMA kernels read 16-channel heads directly), else 32 (fp32 d = 16 is
// padded to 32).
int64_t kernel_d(int64_t d, int dtype) {
  if (d == 64) return 64;
  if (d == 16 && dtype == TRIATTN_BF16) return 16;
  return triattn::HEAD_DIM;
}
// fp32 d = 16 runs on zero-padded 32-channel copies held in the workspace.
bool padded16(int64_t d, int dtype) { return d == 16 && dtype != TRIATTN_BF16; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Row chunks of the bias-gradient reduction over nr rows (at most 16 partial
// slabs).  Each workgroup of the bias-gradient kernel takes 128 queries x 128
// keys of one head over one chunk of rows and fills a CU on its own, so the
// kernel runs in rounds of 256 workgroups.  The cost model, in units of one
// row's work: per round the chunk's rows plus about 3.3 for the workgroup's
// fixed work (bias tile, pipeline fill, slab store), plus about 1 per slab
// for the reduction that reads the slabs back.
int db_row_chunks(int64_t n, int64_t nr, int64_t h) {
  const int64_t tiles = h * ((n + 127) / 128) * ((n + 127) / 128);
  int best = 1;
  double best_cost = 1e300;
  for (int64_t c = 1; c <= 16 && c <= nr; ++c) {
    const int64_t rpc = (nr + c - 1) / c, chunks = (nr + rpc - 1) / rpc;
    const int64_t rounds = (tiles * chunks + 255) / 256;
    const double cost = (double)rounds * ((double)rpc + 3.3) + (double)chunks;
    if (cost < best_cost) {
      best_cost = cost;
      best = (int)chunks;
    }
  }
  return best;
}

struct Layout {
  size_t bt, btT, kbits, rowfull, lse2, dsum, da, dalo, slabs, total;
  int nrc;
};

// Workspace layout for nr rows of pair length n (offsets in bytes, each
// 256-aligned):
//   forward : bt [H][np][np] f32, kbits [nr][np/32] u32, rowfull [nr] u32
//   backward: bt, btT [H][np][np] f32, kbits, rowfull, lse2 and dsum [H][nr][np] f32,
//             dA [nr][n][H][32] dtype (bf16: plus its low part, same size),
//             slabs [nrc][H][np][np] f32
Layout plan(bool bwd, int dtype, int64_t n, int64_t nr, int64_t h, int64_t kd = 32) {
  const size_t np = (size_t)((n + 31) / 32 * 32);
  const size_t plane = (size_t)h * np * np * sizeof(float);
  Layout L{};
  size_t off = 0;
  L.bt = off;
  off += round256(plane);
  if (bwd) {
    L.btT = off;
    off += round256(plane);
  }
  L.kbits = off;
  off += round256((size_t)nr * (np / 32) * sizeof(uint32_t));
  L.rowfull = off;
  off += round256((size_t)nr * sizeof(uint32_t));
  if (bwd) {
    const size_t rows = (size_t)h * nr * np * sizeof(float);
    L.lse2 = off;
    off += round256(rows);
    L.dsum = off;
    off += round256(rows);
    const size_t pair = (size_t)nr * n * h * kd * (dtype == TRIATTN_BF16 ? 2 : 4);
    L.da = off;
    off += round256(pair);
    L.dalo = off;
    if (dtype == TRIATTN_BF16) off += round256(pair);
    L.nrc = db_row_chunks(n, nr, h);
    L.slabs = off;
    off += round256((size_t)L.nrc * plane);
  }
  L.total = off;
  return L;
}

// nr = rows computed: n for a whole call, a row range's length otherwise
// (starting node only; the range's tensors then hold nr rows).
Geom geom(int node, int64_t n, int64_t nr, int64_t h, float scale, int64_t kd = 32) {
  Geom g;
  g.n = (int)n;
  g.nr = (int)nr;
  g.H = (int)h;
  g.np = (int)((n + 31) / 32 * 32);
  g.nkt = g.np / 32;
  g.d = (int)kd;
  const int64_t pos = h * kd, row = n * pos;
  g.sRow = node == TRIATTN_STARTING ? row : pos;
  g.sPos = node == TRIATTN_STARTING ? pos : row;
  g.lRow = node == TRIATTN_STARTING ? n * h : h;
  g.lPos = node == TRIATTN_STARTING ? h : n * h;
  g.scale = scale;
  g.batch = 1;
  g.bPair = g.bBias = g.bMask = g.bWs = 0;
  return g;
}

triattn::Prep prep_ptrs(const Layout& L, void* ws, bool bwd) {
  char* b = (char*)ws;
  return triattn::Prep{(float*)(b + L.bt), bwd ? (float*)(b + L.btT) : nullptr,
                       (uint32_t*)(b + L.kbits), (uint32_t*)(b + L.rowfull)};
}

template <typename T>
int run_fwd(int node, const Geom& g, const Layout& L, const void* q, const void* k,
            const void* v, const void* gate, const void* bias, const uint8_t* mask, void* out,
            float* lse, void* ws, hipStream_t s) {
  const triattn::Prep p = prep_ptrs(L, ws, false);
  if (triattn::launch_prep<T>(g, node, (const T*)bias, mask, p, s) != hipSuccess)
    return TRIATTN_ERR_HIP;
  if (triattn::launch_fwd<T>(g, p, (const T*)q, (const T*)k, (const T*)v, (const T*)gate,
                             (T*)out, lse, s) != hipSuccess)
    return TRIATTN_ERR_HIP;
  return TRIATTN_OK;
}

template <typename T>
int run_bwd(int node, const Geom& g, const Layout& L, const void* q, const void* k,
            const void* v, const void* gate, const void* bias, const uint8_t* mask,
            const void* out, const float* lse, const void* dout, void* dq, void* dk, void* dv,
            void* dg, void* dbias, float* dbias_f32, void* ws, hipStream_t s) {
  const triattn::Prep p = prep_ptrs(L, ws, true);
  char* b = (char*)ws;
  const triattn::BwdWs w{(float*)(b + L.lse2), (float*)(b + L.dsum), (void*)(b + L.da),
                         std::is_same<T, float>::value ? nullptr : (void*)(b + L.dalo),
                         (float*)(b + L.slabs), L.nrc};
  if (triattn::launch_prep<T>(g, node, (const T*)bias, mask, p, s) != hipSuccess)
    return TRIATTN_ERR_HIP;
  if (triattn::launch_bwd<T>(g, node, p, w, (const T*)q, (const T*)k, (const T*)v,
                             (const T*)gate, (const T*)out, lse, (const T*)dout, (T*)dq, (T*)dk,
                             (T*)dv, (T*)dg, (T*)dbias, dbias_f32, s) != hipSuccess)
    return TRIATTN_ERR_HIP;
  return TRIATTN_OK;
}

// Workspace of a whole-map call: the d = 32 layout, then (d = 16) the
// padded copies [n][n][h][32] of q, k, v, g and out (forward) or of q, k, v,
// g, out, dout, dq, dk, dv, dg (backward).
struct Whole {
  Layout L;
  size_t pad0, pad_bytes, total;
};

Whole whole_plan(bool bwd, int dtype, int64_t n, int64_t h, int64_t d) {
  Whole w{plan(bwd, dtype, n, n, h, kernel_d(d, dtype)), 0, 0, 0};
  w.pad0 = w.L.total;
  const int npad = padded16(d, dtype) ? (bwd ? 10 : 5) : 0;
  w.pad_bytes = round256((size_t)n * n * h * triattn::HEAD_DIM * (dtype == TRIATTN_BF16 ? 2 : 4));
  w.total = w.pad0 + (size_t)npad * w.pad_bytes;
  return w;
}

template <typename T>
int fwd_one(int node, const Geom& g, const Whole& W, int64_t d, const void* q, const void* k,
            const void* v, const void* gate, const void* bias, const uint8_t* mask, void* out,
            float* lse, void* ws, hipStream_t s) {
  if (!padded16(d, std::is_same<T, float>::value ? TRIATTN_F32 : TRIATTN_BF16))
    return run_fwd<T>(node, g, W.L, q, k, v, gate, bias, mask, out, lse, ws, s);
  const int64_t rows = (int64_t)g.n * g.n * g.H;
  char* p[5];
  for (int i = 0; i < 5; ++i) p[i] = (char*)ws + W.pad0 + i * W.pad_bytes;
  const void* in[4] = {q, k, v, gate};
  for (int i = 0; i < 4; ++i)
    if (triattn::launch_pad16(in[i], p[i], rows, sizeof(T), s) != hipSuccess)
      return TRIATTN_ERR_HIP;
  const int r = run_fwd<T>(node, g, W.L, p[0], p[1], p[2], p[3], bias, mask, p[4], lse, ws, s);
  if (r != TRIATTN_OK) return r;
  return triattn::launch_unpad16(p[4], out, rows, sizeof(T), s) == hipSuccess ? TRIATTN_OK
                                                                               : TRIATTN_ERR_HIP;
}

template <typename T>
int bwd_one(int node, const Geom& g, const Whole& W, int64_t d, const void* q, const void* k,
            const void* v, const void* gate, const void* bias, const uint8_t* mask,
            const void* out, const float* lse, const void* dout, void* dq, void* dk, void* dv,
            void* dg, void* dbias, void* ws, hipStream_t s) {
  if (!padded16(d, std::is_same<T, float>::value ? TRIATTN_F32 : TRIATTN_BF16))
    return run_bwd<T>(node, g, W.L, q, k, v, gate, bias, mask, out, lse, dout, dq, dk, dv, dg,
                      dbias, nullptr, ws, s);
  const int64_t rows = (int64_t)g.n * g.n * g.H;
  char* p[10];
  for (int i = 0; i < 10; ++i) p[i] = (char*)ws + W.pad0 + i * W.pad_bytes;
  const void* in[6] = {q, k, v, gate, out, dout};
  for (int i = 0; i < 6; ++i)
    if (triattn::launch_pad16(in[i], p[i], rows, sizeof(T), s) != hipSuccess)
      return TRIATTN_ERR_HIP;
  const int r = run_bwd<T>(node, g, W.L, p[0], p[1], p[2], p[3], bias, mask, p[4], lse, p[5],
                           p[6], p[7], p[8], p[9], dbias, nullptr, ws, s);
  if (r != TRIATTN_OK) return r;
  void* outs[4] = {dq, dk, dv, dg};
  for (int i = 0; i < 4; ++i)
    if (triattn::launch_unpad16(p[6 + i], outs[i], rows, sizeof(T), s) != hipSuccess)
      return TRIATTN_ERR_HIP;
  return TRIATTN_OK;
}

}  // namespace

extern "C" {

int tri_attn_fwd_workspace_bytes(int node, int dtype, int64_t n, int64_t h, int64_t d,
                                 size_t* bytes) {
  const int st = check_shape(node, dtype, n, h, d, true);
  if (st != TRIATTN_OK) return st;
  if (bytes == nullptr) return TRIATTN_ERR_INVALID_ARG;
  *bytes = whole_plan(false, dtype, n, h, d).total;
  return TRIATTN_OK;
}

int tri_attn_bwd_workspace_bytes(int node, int dtype, int64_t n, int64_t h, int64_t d,
                                 size_t* bytes) {
  const int st = check_shape(node, dtype, n, h, d, true);
  if (st != TRIATTN_OK) return st;
  if (bytes == nullptr) return TRIATTN_ERR_INVALID_ARG;
  *bytes = whole_plan(true, dtype, n, h, d).total;
  return TRIATTN_OK;
}

int tri_attn_fwd(int node, int dtype, int64_t n, int64_t h, int64_t d, float scale,
                 const void* q, const void* k, const void* v, const void* g, const void* bias,
                 const uint8_t* mask, void* out, float* lse, void* workspace,
                 size_t workspace_bytes, void* stream) {
  int st = check_shape(node, dtype, n, h, d, true);
  if (st != TRIATTN_OK) return st;
  if (!(isfinite(scale) && scale > 0.f)) return TRIATTN_ERR_INVALID_ARG;
  const void* ptrs[] = {q, k, v, g, bias, out, lse};
  for (const void* p : ptrs)
    if (p == nullptr || !aligned16(p)) return TRIATTN_ERR_INVALID_ARG;
  const Whole W = whole_plan(false, dtype, n, h, d);
  if (workspace == nullptr || !aligned16(workspace) || workspace_bytes < W.total)
    return TRIATTN_ERR_WORKSPACE;
  const Geom geo = geom(node, n, n, h, scale, kernel_d(d, dtype));
  hipStream_t s = (hipStream_t)stream;
  if (dtype == TRIATTN_BF16)
    return fwd_one<triattn::bf16>(node, geo, W, d, q, k, v, g, bias, mask, out, lse, workspace,
                                  s);
  return fwd_one<float>(node, geo, W, d, q, k, v, g, bias, mask, out, lse, workspace, s);
}

int tri_attn_bwd(int node, int dtype, int64_t n, int64_t h, int64_t d, float scale,
                 const void* q, const void* k, const void* v, const void* g, const void* bias,
                 const uint8_t* mask, const void* out, const float* lse, const void* dout,
                 void* dq, void* dk, void* dv, void* dg, void* dbias, void* workspace,
                 size_t workspace_bytes, void* stream) {
  int st = check_shape(node, dtype, n, h, d, true);
  if (st != TRIATTN_OK) return st;
  if (!(isfinite(scale) && scale > 0.f)) return TRIATTN_ERR_INVALID_ARG;
  const void* ptrs[] = {q, k, v, g, bias, out, lse, dout, dq, dk, dv, dg, dbias};
  for (const void* p : ptrs)
    if (p == nullptr || !aligned16(p)) return TRIATTN_ERR_INVALID_ARG;
  const Whole W = whole_plan(true, dtype, n, h, d);
  if (workspace == nullptr || !aligned16(workspace) || workspace_bytes < W.total)
    return TRIATTN_ERR_WORKSPACE;
  const Geom geo = geom(node, n, n, h, scale, kernel_d(d, dtype));
  hipStream_t s = (hipStream_t)stream;
  if (dtype == TRIATTN_BF16)
    return bwd_one<triattn::bf16>(node, geo, W, d, q, k, v, g, bias, mask, out, lse, dout, dq,
                                  dk, dv, dg, dbias, workspace, s);
  return bwd_one<float>(node, geo, W, d, q, k, v, g, bias, mask, out, lse, dout, dq, dk, dv, dg,
                        dbias, workspace, s);
}

}  // extern "C"

// ---- the forward for callers that cannot allocate ------------------------------------------
//
// Its workspace (bias planes, key bits) lives in this file-scope device array;
// each GPU the library runs on holds its own copy until the process ends.  In
// host code `scratch` names a host-side stand-in, not the device array: the
// device address comes from hipGetSymbolAddress, looked up once per device
// with that device current, and only that address reaches the kernels.
static __device__ __align__(256) char scratch[TRIATTN_FWD_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[MAX_DEVICES] = {};  // device address of `scratch`, per device

// Device address of this device's scratch array (the stream's device must be
// the current one).
int scratch_address(hipStream_t s, void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return TRIATTN_ERR_HIP;
  if (s != nullptr) {
    hipDevice_t sd = -1;
    if (hipStreamGetDevice(s, &sd) != hipSuccess) return TRIATTN_ERR_HIP;
    if (sd != dev) return TRIATTN_ERR_INVALID_ARG;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_dev[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
      return TRIATTN_ERR_HIP;
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return TRIATTN_OK;
}

}  // namespace

extern "C" {

int tri_attn_fwd_noalloc(int node, int dtype, int64_t n, int64_t h, int64_t d, float scale,
                         const void* q, const void* k, const void* v, const void* g,
                         const void* bias, const uint8_t* mask, void* out, float* lse,
                         void* stream) {
  int st = check_shape(node, dtype, n, h, d, true);
  if (st != TRIATTN_OK) return st;
  if (!(isfinite(scale) && scale > 0.f)) return TRIATTN_ERR_INVALID_ARG;
  const void* ptrs[] = {q, k, v, g, bias, out, lse};
  for (const void* p : ptrs)
    if (p == nullptr || !aligned16(p)) return TRIATTN_ERR_INVALID_ARG;
  const Whole W = whole_plan(false, dtype, n, h, d);
  if (W.total > (size_t)TRIATTN_FWD_NOALLOC_SCRATCH_BYTES) return TRIATTN_ERR_TOO_LARGE;
  hipStream_t s = (hipStream_t)stream;
  void* ws = nullptr;
  st = scratch_address(s, &ws);
  if (st != TRIATTN_OK) return st;
  // every byte of the workspace the forward reads is written first by its
  // preparation kernels (bias planes, key bits), so nothing needs clearing
  const Geom geo = geom(node, n, n, h, scale, kernel_d(d, dtype));
  if (dtype == TRIATTN_BF16)
    return fwd_one<triattn::bf16>(node, geo, W, d, q, k, v, g, bias, mask, out, lse, ws, s);
  return fwd_one<float>(node, geo, W, d, q, k, v, g, bias, mask, out, lse, ws, s);
}

// ---- a batch of pair maps -----------------------------------------------------------------

}  // extern "C"

namespace {

constexpr int64_t MAX_BATCH = (int64_t)1 << 20;

// Per-sample element counts and the checks shared by the batched calls.
struct BatchStrides {
  int64_t pair, bias, lse, mask;  // elements per sample
  size_t el;                      // bytes per dtype element
};

BatchStrides batch_strides(int dtype, int64_t n, int64_t h, int64_t d) {
  return BatchStrides{n * n * h * d, n * n * h, n * n * h, n * n,
                      (size_t)(dtype == TRIATTN_BF16 ? 2 : 4)};
}

// Batched calls run all samples in one launch per kernel (the sample is the
// grid's z index, each sample with its own copy of the workspace) when the
// workspace holds `batch` copies; otherwise, and for fp32 d = 16 (which goes
// through per-sample zero-padded copies), sample by sample.
constexpr int64_t MAX_GRID_BATCH = 65535;  // grid z extent
bool one_grid(int64_t batch, int64_t d, int dtype) {
  return batch > 1 && batch <= MAX_GRID_BATCH && !padded16(d, dtype);
}
size_t batched_bytes(bool bwd, int dtype, int64_t batch, int64_t n, int64_t h, int64_t d) {
  const size_t one = whole_plan(bwd, dtype, n, h, d).total;
  return one_grid(batch, d, dtype) ? (size_t)batch * one : one;
}
// The geometry of a one-launch batch: per-sample strides of the tensors and
// of the workspace.
Geom batched_geom(Geom g, int64_t batch, const BatchStrides& S, bool mask, size_t ws_one) {
  g.batch = (int)batch;
  g.bPair = S.pair;
  g.bBias = S.bias;
  g.bMask = mask ? S.mask : 0;
  g.bWs = (int64_t)ws_one;
  return g;
}

}  // namespace

extern "C" {

int tri_attn_fwd_batched_workspace_bytes(int node, int dtype, int64_t batch, int64_t n,
                                         int64_t h, int64_t d, size_t* bytes) {
  const int st = check_shape(node, dtype, n, h, d, true);
  if (st != TRIATTN_OK) return st;
  if (batch < 1 || batch > MAX_BATCH || bytes == nullptr) return TRIATTN_ERR_INVALID_ARG;
  *bytes = batched_bytes(false, dtype, batch, n, h, d);
  return TRIATTN_OK;
}

int tri_attn_bwd_batched_workspace_bytes(int node, int dtype, int64_t batch, int64_t n,
                                         int64_t h, int64_t d, size_t* bytes) {
  const int st = check_shape(node, dtype, n, h, d, true);
  if (st != TRIATTN_OK) return st;
  if (batch < 1 || batch > MAX_BATCH || bytes == nullptr) return TRIATTN_ERR_INVALID_ARG;
  *bytes = batched_bytes(true, dtype, batch, n, h, d);
  return TRIATTN_OK;
}

int tri_attn_fwd_batched(int node, int dtype, int64_t batch, int64_t n, int64_t h, int64_t d,
                         float scale, const void* q, const void* k, const void* v, const void* g,
                         const void* bias, const uint8_t* mask, void* out, float* lse,
                         void* workspace, size_t workspace_bytes, void* stream) {
  int st = check_shape(node, dtype, n, h, d, true);
  if (st != TRIATTN_OK) return st;
  if (batch < 1 || batch > MAX_BATCH) return TRIATTN_ERR_INVALID_ARG;
  if (!(isfinite(scale) && scale > 0.f)) return TRIATTN_ERR_INVALID_ARG;
  const void* ptrs[] = {q, k, v, g, bias, out, lse};
  for (const void* p : ptrs)
    if (p == nullptr || !aligned16(p)) return TRIATTN_ERR_INVALID_ARG;
  const Whole W = whole_plan(false, dtype, n, h, d);
  if (workspace == nullptr || !aligned16(workspace) || workspace_bytes < W.total)
    return TRIATTN_ERR_WORKSPACE;
  const Geom geo = geom(node, n, n, h, scale, kernel_d(d, dtype));
  const BatchStrides S = batch_strides(dtype, n, h, d);
  hipStream_t s = (hipStream_t)stream;
  if (one_grid(batch, d, dtype) && workspace_bytes / (size_t)batch >= W.total) {
    const Geom gb = batched_geom(geo, batch, S, mask != nullptr, W.total);
    return dtype == TRIATTN_BF16
               ? fwd_one<triattn::bf16>(node, gb, W, d, q, k, v, g, bias, mask, out, lse,
                                        workspace, s)
               : fwd_one<float>(node, gb, W, d, q, k, v, g, bias, mask, out, lse, workspace, s);
  }
  for (int64_t b = 0; b < batch; ++b) {
    const size_t op = (size_t)(b * S.pair) * S.el, ob = (size_t)(b * S.bias) * S.el;
    const uint8_t* mb = mask ? mask + b * S.mask : nullptr;
    float* lb = lse + b * S.lse;
    const int r =
        dtype == TRIATTN_BF16
            ? fwd_one<triattn::bf16>(node, geo, W, d, (const char*)q + op, (const char*)k + op,
                                     (const char*)v + op, (const char*)g + op,
                                     (const char*)bias + ob, mb, (char*)out + op, lb, workspace, s)
            : fwd_one<float>(node, geo, W, d, (const char*)q + op, (const char*)k + op,
                             (const char*)v + op, (const char*)g + op, (const char*)bias + ob, mb,
                             (char*)out + op, lb, workspace, s);
    if (r != TRIATTN_OK) return r;
  }
  return TRIATTN_OK;
}

int tri_attn_bwd_batched(int node, int dtype, int64_t batch, int64_t n, int64_t h, int64_t d,
                         float scale, const void* q, const void* k, const void* v, const void* g,
                         const void* bias, const uint8_t* mask, const void* out,
                         const float* lse, const void* dout, void* dq, void* dk, void* dv,
                         void* dg, void* dbias, void* workspace, size_t workspace_bytes,
                         void* stream) {
  int st = check_shape(node, dtype, n, h, d, true);
  if (st != TRIATTN_OK) return st;
  if (batch < 1 || batch > MAX_BATCH) return TRIATTN_ERR_INVALID_ARG;
  if (!(isfinite(scale) && scale > 0.f)) return TRIATTN_ERR_INVALID_ARG;
  const void* ptrs[] = {q, k, v, g, bias, out, lse, dout, dq, dk, dv, dg, dbias};
  for (const void* p : ptrs)
    if (p == nullptr || !aligned16(p)) return TRIATTN_ERR_INVALID_ARG;
  const Whole W = whole_plan(true, dtype, n, h, d);
  if (workspace == nullptr || !aligned16(workspace) || workspace_bytes < W.total)
    return TRIATTN_ERR_WORKSPACE;
  const Geom geo = geom(node, n, n, h, scale, kernel_d(d, dtype));
  const BatchStrides S = batch_strides(dtype, n, h, d);
  hipStream_t s = (hipStream_t)stream;
  if (one_grid(batch, d, dtype) && workspace_bytes / (size_t)batch >= W.total) {
    const Geom gb = batched_geom(geo, batch, S, mask != nullptr, W.total);
    return dtype == TRIATTN_BF16
               ? bwd_one<triattn::bf16>(node, gb, W, d, q, k, v, g, bias, mask, out, lse, dout,
                                        dq, dk, dv, dg, dbias, workspace, s)
               : bwd_one<float>(node, gb, W, d, q, k, v, g, bias, mask, out, lse, dout, dq, dk,
                                dv, dg, dbias, workspace, s);
  }
  for (int64_t b = 0; b < batch; ++b) {
    const size_t op = (size_t)(b * S.pair) * S.el, ob = (size_t)(b * S.bias) * S.el;
    const uint8_t* mb = mask ? mask + b * S.mask : nullptr;
    const float* lb = lse + b * S.lse;
    auto P = [&](const void* p) { return (const char*)p + op; };
    auto Q = [&](void* p) { return (char*)p + op; };
    const int r =
        dtype == TRIATTN_BF16
            ? bwd_one<triattn::bf16>(node, geo, W, d, P(q), P(k), P(v), P(g),
                                     (const char*)bias + ob, mb, P(out), lb, P(dout), Q(dq), Q(dk),
                                     Q(dv), Q(dg), (char*)dbias + ob, workspace, s)
            : bwd_one<float>(node, geo, W, d, P(q), P(k), P(v), P(g), (const char*)bias + ob, mb,
                             P(out), lb, P(dout), Q(dq), Q(dk), Q(dv), Q(dg), (char*)dbias + ob,
                             workspace, s);
    if (r != TRIATTN_OK) return r;
  }
  return TRIATTN_OK;
}

// ---- starting node over a range of rows -------------------------------------------------

}  // extern "C"

namespace {

int rows_check(int dtype, int64_t n, int64_t rows, int64_t h, int64_t d) {
  const int st = check_shape(TRIATTN_STARTING, dtype, n, h, d);
  if (st != TRIATTN_OK) return st;
  if (rows < 1 || rows > n) return TRIATTN_ERR_INVALID_ARG;
  return TRIATTN_OK;
}

}  // namespace

extern "C" {

int tri_attn_rows_fwd_workspace_bytes(int dtype, int64_t n, int64_t rows, int64_t h, int64_t d,
                                      size_t* bytes) {
  const int st = rows_check(dtype, n, rows, h, d);
  if (st != TRIATTN_OK) return st;
  if (bytes == nullptr) return TRIATTN_ERR_INVALID_ARG;
  *bytes = plan(false, dtype, n, rows, h).total;
  return TRIATTN_OK;
}

int tri_attn_rows_bwd_workspace_bytes(int dtype, int64_t n, int64_t rows, int64_t h, int64_t d,
                                      size_t* bytes) {
  const int st = rows_check(dtype, n, rows, h, d);
  if (st != TRIATTN_OK) return st;
  if (bytes == nullptr) return TRIATTN_ERR_INVALID_ARG;
  *bytes = plan(true, dtype, n, rows, h).total;
  return TRIATTN_OK;
}

int tri_attn_rows_fwd(int dtype, int64_t n, int64_t rows, int64_t h, int64_t d, float scale,
                      const void* q, const void* k, const void* v, const void* g,
                      const void* bias, const uint8_t* mask, void* out, float* lse,
                      void* workspace, size_t workspace_bytes, void* stream) {
  int st = rows_check(dtype, n, rows, h, d);
  if (st != TRIATTN_OK) return st;
  if (!(isfinite(scale) && scale > 0.f)) return TRIATTN_ERR_INVALID_ARG;
  const void* ptrs[] = {q, k, v, g, bias, out, lse};
  for (const void* p : ptrs)
    if (p == nullptr || !aligned16(p)) return TRIATTN_ERR_INVALID_ARG;
  const Layout L = plan(false, dtype, n, rows, h);
  if (workspace == nullptr || !aligned16(workspace) || workspace_bytes < L.total)
    return TRIATTN_ERR_WORKSPACE;
  const Geom geo = geom(TRIATTN_STARTING, n, rows, h, scale);
  hipStream_t s = (hipStream_t)stream;
  if (dtype == TRIATTN_BF16)
    return run_fwd<triattn::bf16>(TRIATTN_STARTING, geo, L, q, k, v, g, bias, mask, out, lse,
                                  workspace, s);
  return run_fwd<float>(TRIATTN_STARTING, geo, L, q, k, v, g, bias, mask, out, lse, workspace,
                        s);
}

int tri_attn_rows_bwd(int dtype, int64_t n, int64_t rows, int64_t h, int64_t d, float scale,
                      const void* q, const void* k, const void* v, const void* g,
                      const void* bias, const uint8_t* mask, const void* out, const float* lse,
                      const void* dout, void* dq, void* dk, void* dv, void* dg,
                      float* dbias_partial, void* workspace, size_t workspace_bytes,
                      void* stream) {
  int st = rows_check(dtype, n, rows, h, d);
  if (st != TRIATTN_OK) return st;
  if (!(isfinite(scale) && scale > 0.f)) return TRIATTN_ERR_INVALID_ARG;
  const void* ptrs[] = {q, k, v, g, bias, out, lse, dout, dq, dk, dv, dg, dbias_partial};
  for (const void* p : ptrs)
    if (p == nullptr || !aligned16(p)) return TRIATTN_ERR_INVALID_ARG;
  const Layout L = plan(true, dtype, n, rows, h);
  if (workspace == nullptr || !aligned16(workspace) || workspace_bytes < L.total)
    return TRIATTN_ERR_WORKSPACE;
  const Geom geo = geom(TRIATTN_STARTING, n, rows, h, scale);
  hipStream_t s = (hipStream_t)stream;
  if (dtype == TRIATTN_BF16)
    return run_bwd<triattn::bf16>(TRIATTN_STARTING, geo, L, q, k, v, g, bias, mask, out, lse,
                                  dout, dq, dk, dv, dg, nullptr, dbias_partial, workspace, s);
  return run_bwd<float>(TRIATTN_STARTING, geo, L, q, k, v, g, bias, mask, out, lse, dout, dq, dk,
                        dv, dg, nullptr, dbias_partial, workspace, s);
}

// ---- fused layer-norm + linear projection ---------------------------------------------

}  // extern "C"

namespace {

int lnl_check(int dtype, int64_t m, int64_t k, int n_out, const int64_t* cols, int64_t* ncols) {
  if (dtype != TRIATTN_F32 && dtype != TRIATTN_BF16) return TRIATTN_ERR_INVALID_ARG;
  if (m < 1 || m > ((int64_t)1 << 31) || k < 1 || n_out < 1 || cols == nullptr)
    return TRIATTN_ERR_INVALID_ARG;
  if (n_out > triattn::LNL_MAX_OUT) return TRIATTN_ERR_UNSUPPORTED;
  int64_t total = 0;
  for (int i = 0; i < n_out; ++i) {
    if (cols[i] < 1) return TRIATTN_ERR_INVALID_ARG;
    if (cols[i] % 4 != 0) return TRIATTN_ERR_UNSUPPORTED;
    total += cols[i];
  }
  if (total > 1024) return TRIATTN_ERR_UNSUPPORTED;
  if (dtype != TRIATTN_BF16 || k != triattn::LNL_K) return TRIATTN_ERR_UNSUPPORTED;
  *ncols = total;
  return TRIATTN_OK;
}

size_t lnl_np(int64_t ncols) { return (size_t)((ncols + 31) / 32 * 32); }

// Where each 32-column tile of o2 (or dO2) lives (see LnlTile).
void lnl_tiles(int64_t m, int64_t ncols, int n_out, const int* start, triattn::bf16* const* ptrs,
               triattn::LnlTile* tile) {
  for (int t = 0; t < (int)((ncols + 31) / 32); ++t) {
    const int col = 32 * t;
    int i = 0;
    while (i + 1 < n_out && col >= start[i + 1]) ++i;
    triattn::LnlTile& e = tile[t];
    e.base = ptrs[i];
    e.off = col - start[i];
    e.w = start[i + 1] - start[i];
    e.fast = (e.off + 32 <= e.w && e.w % 8 == 0 && e.off % 8 == 0 &&
              (uint64_t)(m + 32) * (uint64_t)e.w * 2u < ((uint64_t)1 << 32))
                 ? 1
                 : 0;
  }
}

// Columns per column group of the forward: the fewest groups of at most
// LNL_GROUP columns, balanced, in whole 32-column tiles.
int lnl_group_width(int64_t ncols) {
  const int64_t tiles = (int64_t)lnl_np(ncols) / 32;
  const int64_t groups = (tiles * 32 + triattn::LNL_GROUP - 1) / triattn::LNL_GROUP;
  return (int)((tiles + groups - 1) / groups * 32);
}

}  // namespace

extern "C" {

int tri_ln_linear_fwd(int dtype, int64_t m, int64_t k, int n_out, const int64_t* cols, float eps,
                      const void* x, const void* gamma, const void* beta, const void* w,
                      void* const* outs, float* mean, float* rstd, void* stream) {
  int64_t ncols = 0;
  int st = lnl_check(dtype, m, k, n_out, cols, &ncols);
  if (st != TRIATTN_OK) return st;
  if (!(isfinite(eps) && eps >= 0.f) || outs == nullptr) return TRIATTN_ERR_INVALID_ARG;
  const void* ptrs[] = {x, gamma, beta, w, mean, rstd};
  for (const void* p : ptrs)
    if (p == nullptr || !aligned16(p)) return TRIATTN_ERR_INVALID_ARG;
  for (int i = 0; i < n_out; ++i)
    if (outs[i] == nullptr || !aligned16(outs[i])) return TRIATTN_ERR_INVALID_ARG;
  triattn::LnlArgs a{};
  a.m = m;
  a.ncols = (int)ncols;
  a.gw = lnl_group_width(ncols);
  a.n_out = n_out;
  int64_t c = 0;
  for (int i = 0; i < n_out; ++i) {
    a.start[i] = (int)c;
    a.out[i] = (triattn::bf16*)outs[i];
    c += cols[i];
  }
  for (int i = n_out; i <= triattn::LNL_MAX_OUT; ++i) a.start[i] = (int)ncols;
  a.eps = eps;
  a.x = (const triattn::bf16*)x;
  a.gamma = (const triattn::bf16*)gamma;
  a.beta = (const triattn::bf16*)beta;
  a.mean = mean;
  a.rstd = rstd;
  a.w = (const triattn::bf16*)w;
  lnl_tiles(m, ncols, n_out, a.start, a.out, a.tile);
  if (triattn::launch_lnl_fwd(a, (hipStream_t)stream) != hipSuccess)
    return TRIATTN_ERR_HIP;
  return TRIATTN_OK;
}

}  // extern "C"

namespace {

// Extra limits of the backward: W stays resident in LDS (ncols <= the
// column group) and every tensor's byte range fits a buffer resource.
int lnl_bwd_check(int dtype, int64_t m, int64_t k, int n_out, const int64_t* cols,
                  int64_t* ncols) {
  const int st = lnl_check(dtype, m, k, n_out, cols, ncols);
  if (st != TRIATTN_OK) return st;
  if (*ncols > triattn::LNL_GROUP) return TRIATTN_ERR_UNSUPPORTED;
  int64_t widest = triattn::LNL_K;
  for (int i = 0; i < n_out; ++i) widest = std::max<int64_t>(widest, cols[i]);
  if ((uint64_t)(m + 32) * (uint64_t)widest * 2u >= ((uint64_t)1 << 31))
    return TRIATTN_ERR_UNSUPPORTED;
  return TRIATTN_OK;
}

}  // namespace

extern "C" {

int tri_ln_linear_bwd_workspace_bytes(int dtype, int64_t m, int64_t k, int n_out,
                                      const int64_t* cols, size_t* bytes) {
  int64_t ncols = 0;
  const int st = lnl_bwd_check(dtype, m, k, n_out, cols, &ncols);
  if (st != TRIATTN_OK) return st;
  if (bytes == nullptr) return TRIATTN_ERR_INVALID_ARG;
  *bytes = round256(triattn::lnl_bwd_workspace(m, (int)lnl_np(ncols)));
  return TRIATTN_OK;
}

int tri_ln_linear_bwd(int dtype, int64_t m, int64_t k, int n_out, const int64_t* cols,
                      const void* x, const void* gamma, const void* beta, const void* w,
                      const float* mean, const float* rstd, const void* const* douts, void* dx,
                      float* dw, float* dgamma, float* dbeta, void* workspace,
                      size_t workspace_bytes, void* stream) {
  int64_t ncols = 0;
  int st = lnl_bwd_check(dtype, m, k, n_out, cols, &ncols);
  if (st != TRIATTN_OK) return st;
  if (douts == nullptr) return TRIATTN_ERR_INVALID_ARG;
  const void* ptrs[] = {x, gamma, beta, w, mean, rstd, dx, dw, dgamma, dbeta};
  for (const void* p : ptrs)
    if (p == nullptr || !aligned16(p)) return TRIATTN_ERR_INVALID_ARG;
  for (int i = 0; i < n_out; ++i)
    if (douts[i] == nullptr || !aligned16(douts[i])) return TRIATTN_ERR_INVALID_ARG;
  size_t need = 0;
  tri_ln_linear_bwd_workspace_bytes(dtype, m, k, n_out, cols, &need);
  if (workspace == nullptr || !aligned16(workspace) || workspace_bytes < need)
    return TRIATTN_ERR_WORKSPACE;
  triattn::LnlBwdArgs a{};
  a.m = m;
  a.ncols = (int)ncols;
  a.np = (int)lnl_np(ncols);
  a.n_out = n_out;
  int64_t c = 0;
  for (int i = 0; i < n_out; ++i) {
    a.start[i] = (int)c;
    a.dout[i] = (const triattn::bf16*)douts[i];
    c += cols[i];
  }
  for (int i = n_out; i <= triattn::LNL_MAX_OUT; ++i) a.start[i] = (int)ncols;
  a.x = (const triattn::bf16*)x;
  a.gamma = (const triattn::bf16*)gamma;
  a.beta = (const triattn::bf16*)beta;
  a.w = (const triattn::bf16*)w;
  a.mean = mean;
  a.rstd = rstd;
  a.dx = (triattn::bf16*)dx;
  a.dw = dw;
  a.dgamma = dgamma;
  a.dbeta = dbeta;
  a.nwg = triattn::lnl_bwd_partials(m);
  a.gpart = (float*)workspace;
  a.gsum = a.gpart + (size_t)a.nwg * (triattn::LNL_K + 1) * a.np;
  lnl_tiles(m, ncols, n_out, a.start, (triattn::bf16* const*)a.dout, a.tile);
  if (triattn::launch_lnl_bwd(a, (hipStream_t)stream) != hipSuccess) return TRIATTN_ERR_HIP;
  return TRIATTN_OK;
}

// ---- fused transition layer ---------------------------------------------------------

}  // extern "C"

namespace {

constexpr int64_t TRN_MAX_F = 2048;

int trn_check(int dtype, int64_t m, int64_t c, int64_t f) {
  if (dtype != TRIATTN_F32 && dtype != TRIATTN_BF16) return TRIATTN_ERR_INVALID_ARG;
  if (m < 1 || m > ((int64_t)1 << 31) || c < 1 || f < 1) return TRIATTN_ERR_INVALID_ARG;
  if (dtype != TRIATTN_BF16 || c != triattn::TRN_C || f % triattn::TRN_GROUP != 0 ||
      f > TRN_MAX_F)
    return TRIATTN_ERR_UNSUPPORTED;
  return TRIATTN_OK;
}

struct TrnLayout {
  size_t img, part, gsum, total;
  int nparts;
};

TrnLayout trn_plan(bool bwd, int64_t m, int64_t f) {
  TrnLayout L{};
  const size_t nch = (size_t)(f / triattn::TRN_FC);
  L.img = 0;
  size_t off = round256(nch * (bwd ? triattn::TRN_BWD_IMG : triattn::TRN_FWD_IMG));
  if (bwd) {
    L.nparts = triattn::trn_bwd_parts(m, (int)f);
    L.part = off;
    off += round256((size_t)L.nparts * (size_t)triattn::trn_part_floats((int)f) * sizeof(float));
    L.gsum = off;
    off += round256(((size_t)triattn::TRN_C * 2 * f + 2 * f) * sizeof(float));
  }
  L.total = off;
  return L;
}

}  // namespace

extern "C" {

int tri_transition_fwd_workspace_bytes(int dtype, int64_t m, int64_t c, int64_t f,
                                       size_t* bytes) {
  const int st = trn_check(dtype, m, c, f);
  if (st != TRIATTN_OK) return st;
  if (bytes == nullptr) return TRIATTN_ERR_INVALID_ARG;
  *bytes = trn_plan(false, m, f).total;
  return TRIATTN_OK;
}

int tri_transition_bwd_workspace_bytes(int dtype, int64_t m, int64_t c, int64_t f,
                                       size_t* bytes) {
  const int st = trn_check(dtype, m, c, f);
  if (st != TRIATTN_OK) return st;
  if (bytes == nullptr) return TRIATTN_ERR_INVALID_ARG;
  *bytes = trn_plan(true, m, f).total;
  return TRIATTN_OK;
}

int tri_transition_fwd(int dtype, int64_t m, int64_t c, int64_t f, float eps, const void* x,
                       const void* gamma, const void* beta, const void* w1, const void* w2,
                       void* out, float* mean, float* rstd, void* workspace,
                       size_t workspace_bytes, void* stream) {
  int st = trn_check(dtype, m, c, f);
  if (st != TRIATTN_OK) return st;
  if (!(isfinite(eps) && eps >= 0.f)) return TRIATTN_ERR_INVALID_ARG;
  const void* ptrs[] = {x, gamma, beta, w1, w2, out, mean, rstd};
  for (const void* p : ptrs)
    if (p == nullptr || !aligned16(p)) return TRIATTN_ERR_INVALID_ARG;
  const TrnLayout L = trn_plan(false, m, f);
  if (workspace == nullptr || !aligned16(workspace) || workspace_bytes < L.total)
    return TRIATTN_ERR_WORKSPACE;
  triattn::TrnFwdArgs a{};
  a.m = m;
  a.f = (int)f;
  a.eps = eps;
  a.x = (const triattn::bf16*)x;
  a.gamma = (const triattn::bf16*)gamma;
  a.beta = (const triattn::bf16*)beta;
  a.w1 = (const triattn::bf16*)w1;
  a.w2 = (const triattn::bf16*)w2;
  a.img = (char*)workspace + L.img;
  a.out = (triattn::bf16*)out;
  a.mean = mean;
  a.rstd = rstd;
  return triattn::launch_trn_fwd(a, (hipStream_t)stream) == hipSuccess ? TRIATTN_OK
                                                                        : TRIATTN_ERR_HIP;
}

int tri_transition_bwd(int dtype, int64_t m, int64_t c, int64_t f, const void* x,
                       const void* gamma, const void* beta, const void* w1, const void* w2,
                       const float* mean, const float* rstd, const void* dout, void* dx,
                       float* dw1, float* dw2, float* dgamma, float* dbeta, void* workspace,
                       size_t workspace_bytes, void* stream) {
  int st = trn_check(dtype, m, c, f);
  if (st != TRIATTN_OK) return st;
  const void* ptrs[] = {x, gamma, beta, w1, w2, mean, rstd, dout, dx, dw1, dw2, dgamma, dbeta};
  for (const void* p : ptrs)
    if (p == nullptr || !aligned16(p)) return TRIATTN_ERR_INVALID_ARG;
  const TrnLayout L = trn_plan(true, m, f);
  if (workspace == nullptr || !aligned16(workspace) || workspace_bytes < L.total)
    return TRIATTN_ERR_WORKSPACE;
  triattn::TrnBwdArgs a{};
  a.m = m;
  a.f = (int)f;
  a.x = (const triattn::bf16*)x;
  a.gamma = (const triattn::bf16*)gamma;
  a.beta = (const triattn::bf16*)beta;
  a.w1 = (const triattn::bf16*)w1;
  a.w2 = (const triattn::bf16*)w2;
  a.mean = mean;
  a.rstd = rstd;
  a.dout = (const triattn::bf16*)dout;
  a.dx = (triattn::bf16*)dx;
  a.dw1 = dw1;
  a.dw2 = dw2;
  a.dgamma = dgamma;
  a.dbeta = dbeta;
  char* b = (char*)workspace;
  a.img = b + L.img;
  a.part = (float*)(b + L.part);
  a.gsum = (float*)(b + L.gsum);
  a.nparts = L.nparts;
  return triattn::launch_trn_bwd(a, (hipStream_t)stream) == hipSuccess ? TRIATTN_OK
                                                                        : TRIATTN_ERR_HIP;
}

const char* tri_attn_status_string(int status) {
  switch (status) {
    case TRIATTN_OK: return "ok";
    case TRIATTN_ERR_INVALID_ARG: return "invalid argument";
    case TRIATTN_ERR_UNSUPPORTED: return "unsupported argument value";
    case TRIATTN_ERR_WORKSPACE: return "workspace missing or too small";
    case TRIATTN_ERR_HIP: return "HIP launch error";
    case TRIATTN_ERR_TOO_LARGE:
      return "problem needs more scratch memory than the allocation-free entry point holds";
    default: return "unknown status";
  }
}

}  // extern "C"
