// jl_api.cpp -- host side of libjetlong.so: the C ABI declared in
// include/jetlong.h.  Validates every argument before anything is launched,
// owns the per-device cache of RoPE cos/sin tables, and dispatches the
// gfx950 kernels.  See the header for the contract of each entry point.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <algorithm>
#include <atomic>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/jetlong.h"

namespace jl {
// kernels (prefill.hip, decode.hip, aux.hip)
size_t prefill_workspace_bytes(bool bifocal, int B, int Hkv, int L);
hipError_t launch_prefill_chunk(bool bifocal, const uint16_t* q, const uint16_t* k,
                                const uint16_t* v, uint16_t* o, float* lse, const float2* table,
                                const float2* rtable, const uint32_t* table16,
                                const uint32_t* rtable16, int freq_map, int B, int Hq, int Hkv,
                                int L, int q_start, int Lq, int kv_stride, int G, int w0,
                                float slack, void* ws, hipStream_t stream, hipEvent_t ev0,
                                hipEvent_t ev1, const int32_t* block_table, int max_pages,
                                int page_shift, int n_pages);
size_t prefill_varlen_workspace_bytes(bool bifocal, int B, int T, int Hq, int Hkv, bool freq);
hipError_t launch_prefill_varlen(bool bifocal, const uint16_t* q, const uint16_t* k,
                                 const uint16_t* v, uint16_t* o, float* lse, const float2* table,
                                 const uint32_t* table16, const int32_t* cu, int B, int T,
                                 int max_len, int Hq, int Hkv,
                                 int w_pre, int w0, float slack, void* ws, hipStream_t stream,
                                 hipEvent_t ev0, hipEvent_t ev1, const double* freq_og);
size_t literal_workspace_bytes(int B, int Hq, int Hkv, int L);
hipError_t launch_prefill_literal(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                  uint16_t* o, float* lse, const float2* table,
                                  const float2* rtable, const uint32_t* table16,
                                  const uint32_t* rtable16, int freq_map, int B, int Hq, int Hkv,
                                  int L, int G, int w0, float slack, void* ws,
                                  hipStream_t stream);
int prefill_rows_per_block();
int prefill_block_q(int g);
int prefill_block_k();
size_t decode_workspace_bytes(int B, int Hq, int Hkv, int max_len);
size_t decode_map_workspace_bytes(int B, int Hq, int Hkv, int max_len, bool freq);
hipError_t launch_decode(bool bifocal, const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                         const int32_t* kv_lens, int max_len, uint16_t* o, const float2* table,
                         int B, int Hq, int Hkv, int w_pre, int w0, float* ws,
                         hipStream_t stream, hipEvent_t ev0, hipEvent_t ev1,
                         const int32_t* block_table, int max_pages, int n_pages, int page_shift,
                         const double* freq_og);
int noalloc_decode_max_len();
size_t noalloc_decode_state_bytes();
hipError_t noalloc_decode_buffers(double theta, const double* omega, hipStream_t stream,
                                  const float2** table, float** states);
hipError_t launch_build_table(float2* table, uint32_t* table16, int n_pos, const double* omega,
                              hipStream_t stream);
hipError_t launch_debug_schedule(const int32_t* lengths, int nl, const int32_t* positions, int np,
                                 int w, int32_t* gout, int32_t* fout, int32_t* dout,
                                 hipStream_t stream);
hipError_t launch_debug_tiles(int L, int BQ, int BK, int w0, int nqb, int nkt, int8_t* out,
                              hipStream_t stream);
}  // namespace jl

namespace {

constexpr int kHeadDim = 128;
constexpr int kDecodeMaxLen = 1 << 23;
// paged chunked prefill: a page holds whole 64-key tiles, and one sequence's
// page list fits the attention kernel's LDS table
constexpr int kPagedPrefillMinPage = 64;
constexpr int kPagedPrefillMaxPages = 4096;  // 512-byte table rows, 32-bit offsets
thread_local std::string t_detail;
// how far (log2 units) a prefill tile's score maximum may lie from the softmax
// reference before the reference moves; the debug entry lowers it so tests
// can drive the rescale path on ordinary data
std::atomic<double> g_rescale_log2{64.0};
// benchmark timing hook: events recorded around the prefill attention kernel
// ([0]) and the decode split kernel ([1]); null when unset
std::mutex g_ev_mu;
hipEvent_t g_events[2][2] = {{nullptr, nullptr}, {nullptr, nullptr}};

void timing_events(int which, hipEvent_t* ev0, hipEvent_t* ev1) {
  std::lock_guard<std::mutex> lock(g_ev_mu);
  *ev0 = g_events[which][0];
  *ev1 = g_events[which][1];
}

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  t_detail = buf;
  return status;
}

int ok() {
  t_detail.clear();
  return JL_OK;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(JL_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return p != nullptr && (reinterpret_cast<uintptr_t>(p) & 15) == 0; }
bool aligned4(const void* p) { return p != nullptr && (reinterpret_cast<uintptr_t>(p) & 3) == 0; }

// ------------------------------------------------------------ table cache
// A table of cap positions is one allocation: cap x 64 fp32 (cos, sin) pairs
// (512 B per position), then the same pairs in fp16, one 32-bit word each
// (256 B per position).
struct TableEntry {
  int device;
  double theta;
  int cap;  // positions held
  float2* ptr;
};
std::mutex g_mu;
std::vector<TableEntry> g_tables;
std::vector<std::pair<int, float2*>> g_retired;  // superseded base tables, freed by jl_release_caches

size_t table_bytes(long long cap) { return (size_t)cap * 64 * (sizeof(float2) + sizeof(uint32_t)); }
const uint32_t* table16_of(const float2* p, long long cap) {
  return reinterpret_cast<const uint32_t*>(p + (size_t)cap * 64);
}

struct Tables {
  const float2* f32;
  const uint32_t* f16;
};

// Returns device tables covering positions [0, n_pos) for the current device.
// A larger request doubles the capacity (waiting for the stream once); the
// superseded table is kept until jl_release_caches (calls in flight on other
// streams may still read it), so the retired total stays below the live one.
// omega_i = theta^(-2i/d), i < d/2 (Sec. 2, the RoPE frequencies)
void rope_omega(double theta, double* omega) {
  for (int i = 0; i < kHeadDim / 2; ++i) omega[i] = std::pow(theta, -2.0 * i / (double)kHeadDim);
}

int get_table(double theta, int n_pos, hipStream_t stream, Tables* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::lock_guard<std::mutex> lock(g_mu);
  TableEntry* found = nullptr;
  for (auto& t : g_tables)
    if (t.device == dev && t.theta == theta) found = &t;
  if (found && found->cap >= n_pos) {
    *out = Tables{found->ptr, table16_of(found->ptr, found->cap)};
    return JL_OK;
  }
  long long cap = 4096;
  while (cap < n_pos) cap *= 2;
  if (found && cap < 2LL * found->cap) cap = 2LL * found->cap;
  if (cap > (1LL << 30) / 64) cap = n_pos;  // keep the element count in range
  float2* p = nullptr;
  e = hipMalloc(&p, table_bytes(cap));
  if (e != hipSuccess) return hip_fail(e, "hipMalloc(rope table)");
  double omega[kHeadDim / 2];
  rope_omega(theta, omega);
  e = jl::launch_build_table(p, const_cast<uint32_t*>(table16_of(p, cap)), (int)cap, omega, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);  // usable from any stream afterwards
  if (e != hipSuccess) {
    (void)hipFree(p);
    return hip_fail(e, "building rope table");
  }
  if (found) {
    g_retired.emplace_back(found->device, found->ptr);
    found->ptr = p;
    found->cap = (int)cap;
  } else {
    g_tables.push_back(TableEntry{dev, theta, (int)cap, p});
  }
  *out = Tables{p, table16_of(p, cap)};
  return JL_OK;
}

// Remote-view frequencies of the frequency-interpolation map (Sec. 4.5, the
// ablation that keeps positions and rescales frequencies, YaRN style): with
// s = max(1, L / w_pretrained), pair i of wavelength lambda_i = 2 pi / omega_i
// completes r_i = w_pretrained / lambda_i turns over the pretraining window;
// gamma_i = clamp((r_i - 1) / (32 - 1), 0, 1) and
// omega'_i = (1 - gamma_i) omega_i / s + gamma_i omega_i.  Fast pairs keep
// their frequency, slow pairs are divided by s.
// omega_i and the ramp gamma_i of pair i (og[0..63], og[64..127]); only the
// factor s depends on the length.
void freq_map_ramp(double theta, int w_pre, double* og) {
  const double kAlpha = 1.0, kBeta = 32.0;
  const double two_pi = 2.0 * std::acos(-1.0);
  for (int i = 0; i < 64; ++i) {
    const double omega = std::pow(theta, -2.0 * i / (double)kHeadDim);
    const double r = (double)w_pre / (two_pi / omega);
    og[i] = omega;
    og[64 + i] = std::min(1.0, std::max(0.0, (r - kAlpha) / (kBeta - kAlpha)));
  }
}

void freq_map_omegas(double theta, int L, int w_pre, double* out) {
  double og[128];
  freq_map_ramp(theta, w_pre, og);
  const double s = std::max(1.0, (double)L / (double)w_pre);
  for (int i = 0; i < 64; ++i) out[i] = (1.0 - og[64 + i]) * og[i] / s + og[64 + i] * og[i];
}

// One frequency-map table per device, for the last (theta, L, w_pretrained)
// used: [L][64] (cos, sin) of p * omega'_i (fp32, then bf16 pairs as in the base
// table), held in a buffer of cap >= L positions.  A new configuration that
// fits is rebuilt in place; one that does not replaces the buffer with one of
// at least twice the capacity.  Either way the device is synchronised first,
// since calls on any stream may still read the old contents: nothing is
// retired, so repeated calls with new lengths keep one buffer per device.
struct FreqTable {
  int device;
  double theta;
  int L, w_pre;
  long long cap;
  float2* ptr;
};
std::vector<FreqTable> g_freq_tables;

int get_freq_table(double theta, int L, int w_pre, hipStream_t stream, Tables* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::lock_guard<std::mutex> lock(g_mu);
  FreqTable* found = nullptr;
  for (auto& t : g_freq_tables)
    if (t.device == dev) found = &t;
  if (found && found->theta == theta && found->L == L && found->w_pre == w_pre) {
    *out = Tables{found->ptr, table16_of(found->ptr, found->cap)};
    return JL_OK;
  }
  if (found) {
    e = hipDeviceSynchronize();  // every earlier call that reads the old table is done
    if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
  }
  float2* p = found ? found->ptr : nullptr;
  long long cap = found ? found->cap : 0;
  if (cap < L) {
    const long long want = std::max<long long>(L, 2 * cap);
    float2* q = nullptr;
    e = hipMalloc(&q, table_bytes(want));
    if (e != hipSuccess) return hip_fail(e, "hipMalloc(frequency-map table)");
    if (p != nullptr) (void)hipFree(p);
    p = q;
    cap = want;
    if (found) {
      found->ptr = p;
      found->cap = cap;
      found->L = -1;  // contents not valid until the build below succeeds
    }
  }
  double omega[64];
  freq_map_omegas(theta, L, w_pre, omega);
  e = jl::launch_build_table(p, const_cast<uint32_t*>(table16_of(p, cap)), L, omega, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) {
    if (found) found->L = -1;
    else (void)hipFree(p);
    return hip_fail(e, "building frequency-map table");
  }
  if (found) {
    found->theta = theta;
    found->L = L;
    found->w_pre = w_pre;
  } else {
    g_freq_tables.push_back(FreqTable{dev, theta, L, w_pre, cap, p});
  }
  *out = Tables{p, table16_of(p, cap)};
  return JL_OK;
}

// ------------------------------------------- prefill scratch, per stream
// The prefill writes each call's rotated K (one image per view) and
// transposed V to scratch before its attention kernel reads them.  One buffer
// per (device, stream): calls on one stream are ordered, so they can share
// it; a call that needs more waits for its stream before replacing it.
struct Scratch {
  int device;
  hipStream_t stream;
  size_t bytes;
  void* ptr;
};
std::vector<Scratch> g_scratch;
std::mutex g_prefill_mu;  // held from scratch lookup to launch, so a concurrent
                          // call on the same stream cannot replace a buffer in between

int get_scratch(hipStream_t stream, size_t bytes, void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::lock_guard<std::mutex> lock(g_mu);
  Scratch* found = nullptr;
  for (auto& sc : g_scratch)
    if (sc.device == dev && sc.stream == stream) found = &sc;
  if (found && found->bytes >= bytes) {
    *out = found->ptr;
    return JL_OK;
  }
  if (found) {
    e = hipStreamSynchronize(stream);  // earlier calls on this stream may still read it
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    (void)hipFree(found->ptr);
    found->ptr = nullptr;
    found->bytes = 0;
  }
  const size_t want = bytes + bytes / 8;  // some room for growth
  void* p = nullptr;
  e = hipMalloc(&p, want);
  if (e != hipSuccess) return hip_fail(e, "hipMalloc(prefill scratch)");
  if (found) {
    found->ptr = p;
    found->bytes = want;
  } else {
    g_scratch.push_back(Scratch{dev, stream, want, p});
  }
  *out = p;
  return JL_OK;
}

int check_common(int B, int Hq, int Hkv, int head_dim, double theta) {
  if (B < 1 || Hq < 1 || Hkv < 1)
    return fail(JL_ERR_INVALID_ARG, "B, Hq, Hkv must be >= 1 (got %d, %d, %d)", B, Hq, Hkv);
  if (Hq % Hkv != 0)
    return fail(JL_ERR_INVALID_ARG, "Hq (%d) must be a multiple of Hkv (%d)", Hq, Hkv);
  if (head_dim < 2 || head_dim % 2 != 0)
    return fail(JL_ERR_INVALID_ARG, "head_dim must be even and >= 2 (got %d)", head_dim);
  if (head_dim != kHeadDim)
    return fail(JL_ERR_UNSUPPORTED, "head_dim %d not built (only 128)", head_dim);
  if (!(theta > 0.0) || !std::isfinite(theta))
    return fail(JL_ERR_INVALID_ARG, "rope_theta must be finite and > 0");
  return JL_OK;
}

// literal: run Eq. (7) as three window passes plus a merge, in the caller's
// workspace (ws, ws_bytes), or at G == 1 the vanilla kernel with its tile
// images in that workspace's tile region; otherwise the fused or vanilla
// kernel with the library scratch.
int prefill_common(bool bifocal, const void* q, const void* k, const void* v, void* o, float* lse,
                   int B, int Hq, int Hkv, int L, int head_dim, double theta, int w_pre, int w0,
                   void* stream, bool literal = false, void* ws = nullptr, size_t ws_bytes = 0,
                   int remote_map = JL_REMOTE_ALIAS, int q_start = 0, int Lq = -1,
                   int kv_stride = -1, const int32_t* block_table = nullptr, int max_pages = 0,
                   int page_shift = 0, int n_pages = 0) {
  // a chunk: queries q_start .. q_start + Lq - 1 over keys [0, L) of a cache
  // with kv_stride rows per sequence; the full prefill has Lq = kv_stride = L
  if (Lq < 0) Lq = L;
  if (kv_stride < 0) kv_stride = L;
  int st = check_common(B, Hq, Hkv, head_dim, theta);
  if (st != JL_OK) return st;
  if (remote_map != JL_REMOTE_ALIAS && remote_map != JL_REMOTE_FREQ)
    return fail(JL_ERR_INVALID_ARG, "remote_map must be JL_REMOTE_ALIAS or JL_REMOTE_FREQ (got %d)",
                remote_map);
  if (L < 1) return fail(JL_ERR_INVALID_ARG, "L must be >= 1 (got %d)", L);
  if (bifocal && w_pre < 1)
    return fail(JL_ERR_INVALID_ARG, "w_pretrained must be >= 1 (got %d)", w_pre);
  if (bifocal && w0 < 0) return fail(JL_ERR_INVALID_ARG, "w_local must be >= 0 (got %d)", w0);
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o))
    return fail(JL_ERR_INVALID_ARG, "q, k, v, o must be non-null and 16-byte aligned");
  if (lse != nullptr && !aligned4(lse)) return fail(JL_ERR_INVALID_ARG, "lse must be 4-byte aligned");
  const int g = Hq / Hkv;
  const int rows = jl::prefill_rows_per_block();
  if (rows % g != 0)
    return fail(JL_ERR_UNSUPPORTED, "GQA group Hq/Hkv = %d must divide %d", g, rows);
  const long long nqb = (Lq + (rows / g) - 1) / (rows / g);
  if (nqb * B * Hkv > 0x7fffffffLL) return fail(JL_ERR_INVALID_ARG, "problem too large");
  if ((long long)B * Hkv > 65535) return fail(JL_ERR_INVALID_ARG, "B * Hkv too large");
  if (literal) {
    const size_t need = jl::literal_workspace_bytes(B, Hq, Hkv, L);
    if (ws == nullptr || ws_bytes < need)
      return fail(JL_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, ws_bytes);
    if ((reinterpret_cast<uintptr_t>(ws) & 255) != 0)
      return fail(JL_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  }
  const int G = bifocal ? (int)jl_group_size(L, w_pre) : 1;
  Tables tab{};
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  st = get_table(theta, L, s, &tab);
  if (st != JL_OK) return st;
  // G == 1: f is the identity and the method is the base model (Sec. 3), so
  // the bifocal entry runs the vanilla kernel and matches it bit for bit.
  // The frequency map's factor s = L / w_pretrained is 1 exactly then too.
  const bool use_bifocal = bifocal && G > 1;
  const int freq_map = remote_map == JL_REMOTE_FREQ ? 1 : 0;
  Tables rtab{};
  if (use_bifocal && freq_map) {
    st = get_freq_table(theta, L, w_pre, s, &rtab);
    if (st != JL_OK) return st;
  }
  const float slack = (float)g_rescale_log2.load();
  if (literal) {
    if (use_bifocal) {
      hipError_t e = jl::launch_prefill_literal((const uint16_t*)q, (const uint16_t*)k,
                                                (const uint16_t*)v, (uint16_t*)o, lse, tab.f32,
                                                rtab.f32, tab.f16, rtab.f16, freq_map, B, Hq,
                                                Hkv, L, G, w0, slack, ws, s);
      if (e != hipSuccess) return hip_fail(e, "literal prefill launch");
      return ok();
    }
  }
  std::lock_guard<std::mutex> launch_lock(g_prefill_mu);
  void* scratch = nullptr;
  if (literal) {
    // the literal workspace ends with the tile images and rerun list that
    // the vanilla kernel needs (the same layout as the library scratch)
    const size_t tail = jl::prefill_workspace_bytes(false, B, Hkv, L);
    scratch = static_cast<char*>(ws) + (jl::literal_workspace_bytes(B, Hq, Hkv, L) - tail);
  } else {
    st = get_scratch(s, jl::prefill_workspace_bytes(use_bifocal, B, Hkv, L), &scratch);
    if (st != JL_OK) return st;
  }
  hipEvent_t ev0, ev1;
  timing_events(0, &ev0, &ev1);
  hipError_t e = jl::launch_prefill_chunk(use_bifocal, (const uint16_t*)q, (const uint16_t*)k,
                                          (const uint16_t*)v, (uint16_t*)o, lse, tab.f32, rtab.f32,
                                          tab.f16, rtab.f16, freq_map, B, Hq, Hkv, L, q_start, Lq,
                                          kv_stride, G, w0, slack, scratch, s, ev0, ev1,
                                          block_table, max_pages, page_shift, n_pages);
  if (e != hipSuccess) return hip_fail(e, "prefill launch");
  return ok();
}

// Packed batch of B sequences, cu_seqlens (device, B + 1) delimiting their
// rows of the T-row tensors; every sequence is prefilled with its own length.
int prefill_varlen(bool bifocal, const void* q, const void* k, const void* v, void* o, float* lse,
                   const int32_t* cu, int B, int T, int max_seqlen, int Hq, int Hkv,
                   int head_dim, double theta, int w_pre, int w0, void* stream,
                   int remote_map = JL_REMOTE_ALIAS) {
  int st = check_common(B, Hq, Hkv, head_dim, theta);
  if (st != JL_OK) return st;
  if (remote_map != JL_REMOTE_ALIAS && remote_map != JL_REMOTE_FREQ)
    return fail(JL_ERR_INVALID_ARG, "remote_map must be JL_REMOTE_ALIAS or JL_REMOTE_FREQ (got %d)",
                remote_map);
  const bool freq = bifocal && remote_map == JL_REMOTE_FREQ;
  if (T < 1) return fail(JL_ERR_INVALID_ARG, "total_tokens must be >= 1 (got %d)", T);
  if (max_seqlen < 1)
    return fail(JL_ERR_INVALID_ARG, "max_seqlen must be >= 1 (got %d)", max_seqlen);
  if (bifocal && w_pre < 1)
    return fail(JL_ERR_INVALID_ARG, "w_pretrained must be >= 1 (got %d)", w_pre);
  if (bifocal && w0 < 0) return fail(JL_ERR_INVALID_ARG, "w_local must be >= 0 (got %d)", w0);
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o))
    return fail(JL_ERR_INVALID_ARG, "q, k, v, o must be non-null and 16-byte aligned");
  if (lse != nullptr && !aligned4(lse)) return fail(JL_ERR_INVALID_ARG, "lse must be 4-byte aligned");
  if (!aligned4(cu)) return fail(JL_ERR_INVALID_ARG, "cu_seqlens must be non-null and aligned");
  const int g = Hq / Hkv;
  const int rows = jl::prefill_rows_per_block();
  if (rows % g != 0)
    return fail(JL_ERR_UNSUPPORTED, "GQA group Hq/Hkv = %d must divide %d", g, rows);
  const long long nq = ((long long)T + rows / g - 1) / (rows / g) + B;
  if (nq * Hkv > 0x7fffffffLL || Hkv > 65535)
    return fail(JL_ERR_INVALID_ARG, "problem too large");
  const int max_len = std::min(max_seqlen, T);  // no sequence is longer than T
  Tables tab{};
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  st = get_table(theta, max_len, s, &tab);
  if (st != JL_OK) return st;
  const float slack = (float)g_rescale_log2.load();
  std::lock_guard<std::mutex> launch_lock(g_prefill_mu);
  void* scratch = nullptr;
  st = get_scratch(s, jl::prefill_varlen_workspace_bytes(bifocal, B, T, Hq, Hkv, freq), &scratch);
  if (st != JL_OK) return st;
  double og[128];
  if (freq) freq_map_ramp(theta, w_pre, og);
  hipEvent_t ev0, ev1;
  timing_events(0, &ev0, &ev1);
  hipError_t e = jl::launch_prefill_varlen(bifocal, (const uint16_t*)q, (const uint16_t*)k,
                                           (const uint16_t*)v, (uint16_t*)o, lse, tab.f32, tab.f16,
                                           cu, B, T,
                                           max_len, Hq, Hkv, w_pre, w0, slack, scratch, s, ev0,
                                           ev1, freq ? og : nullptr);
  if (e != hipSuccess) return hip_fail(e, "varlen prefill launch");
  return ok();
}

// block_table != nullptr: paged pools (kc, vc [n_pages][page_size][Hkv][128],
// max_len = max_pages * page_size); else dense caches [B][max_len][Hkv][128]
int decode_common(bool bifocal, const void* q, const void* kc, const void* vc,
                  const int32_t* kv_lens, int max_len, void* o, int B, int Hq, int Hkv,
                  int head_dim, double theta, int w_pre, int w0, void* ws, size_t ws_bytes,
                  void* stream, const int32_t* block_table = nullptr, int max_pages = 0,
                  int page_size = 0, int n_pages = 0, int remote_map = JL_REMOTE_ALIAS,
                  bool noalloc = false) {
  int page_shift = 0;
  if (remote_map != JL_REMOTE_ALIAS && remote_map != JL_REMOTE_FREQ)
    return fail(JL_ERR_INVALID_ARG, "remote_map must be JL_REMOTE_ALIAS or JL_REMOTE_FREQ (got %d)",
                remote_map);
  const bool freq = bifocal && remote_map == JL_REMOTE_FREQ;
  if (block_table != nullptr) {
    if (!aligned4(block_table))
      return fail(JL_ERR_INVALID_ARG, "block_table must be 4-byte aligned");
    if (page_size < 16 || page_size > (1 << 20) || (page_size & (page_size - 1)) != 0)
      return fail(JL_ERR_INVALID_ARG, "page_size must be a power of two in [16, 2^20] (got %d)",
                  page_size);
    if (max_pages < 1 || n_pages < 1)
      return fail(JL_ERR_INVALID_ARG, "max_pages and n_pages must be >= 1 (got %d, %d)",
                  max_pages, n_pages);
    if ((long long)max_pages * page_size > 0x7fffffffLL)
      return fail(JL_ERR_INVALID_ARG, "max_pages * page_size too large");
    while ((1 << page_shift) < page_size) ++page_shift;
    max_len = max_pages * page_size;
  }
  int st = check_common(B, Hq, Hkv, head_dim, theta);
  if (st != JL_OK) return st;
  if (max_len < 1) return fail(JL_ERR_INVALID_ARG, "max_len must be >= 1 (got %d)", max_len);
  // the split kernel addresses cos/sin table rows with 32-bit byte offsets
  if (max_len > kDecodeMaxLen)
    return fail(JL_ERR_UNSUPPORTED, "decode max_len %d exceeds %d positions", max_len,
                kDecodeMaxLen);
  if (bifocal && w_pre < 1)
    return fail(JL_ERR_INVALID_ARG, "w_pretrained must be >= 1 (got %d)", w_pre);
  if (bifocal && w0 < 0) return fail(JL_ERR_INVALID_ARG, "w_local must be >= 0 (got %d)", w0);
  if (!aligned16(q) || !aligned16(kc) || !aligned16(vc) || !aligned16(o))
    return fail(JL_ERR_INVALID_ARG, "q, k_cache, v_cache, o must be non-null and 16-byte aligned");
  if (!aligned4(kv_lens)) return fail(JL_ERR_INVALID_ARG, "kv_lens must be non-null and aligned");
  if (Hq / Hkv > 8) return fail(JL_ERR_UNSUPPORTED, "decode GQA group %d > 8", Hq / Hkv);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (noalloc) {  // the fixed scratch: bounded sizes, no allocation, no timing events
    if (max_len > jl::noalloc_decode_max_len())
      return fail(JL_ERR_UNSUPPORTED, "no-alloc decode: max_len %d exceeds %d", max_len,
                  jl::noalloc_decode_max_len());
    const size_t states = jl::decode_workspace_bytes(B, Hq, Hkv, max_len);
    if (states > jl::noalloc_decode_state_bytes())
      return fail(JL_ERR_UNSUPPORTED, "no-alloc decode: %zu bytes of split states exceed %zu",
                  states, jl::noalloc_decode_state_bytes());
    double omega[kHeadDim / 2];
    rope_omega(theta, omega);
    const float2* table = nullptr;
    float* st_ws = nullptr;
    hipError_t e = jl::noalloc_decode_buffers(theta, omega, s, &table, &st_ws);
    if (e != hipSuccess) return hip_fail(e, "no-alloc decode scratch");
    e = jl::launch_decode(bifocal, (const uint16_t*)q, (const uint16_t*)kc, (const uint16_t*)vc,
                          kv_lens, max_len, (uint16_t*)o, table, B, Hq, Hkv, w_pre, w0, st_ws, s,
                          nullptr, nullptr, block_table, max_pages, n_pages, page_shift, nullptr);
    if (e != hipSuccess) return hip_fail(e, "decode launch");
    return ok();
  }
  const size_t need = jl::decode_map_workspace_bytes(B, Hq, Hkv, max_len, freq);
  if (ws == nullptr || ws_bytes < need)
    return fail(JL_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, ws_bytes);
  if (!aligned16(ws)) return fail(JL_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
  Tables tab{};
  st = get_table(theta, max_len, s, &tab);
  if (st != JL_OK) return st;
  double og[128];
  if (freq) freq_map_ramp(theta, w_pre, og);
  hipEvent_t ev0, ev1;
  timing_events(1, &ev0, &ev1);
  hipError_t e = jl::launch_decode(bifocal, (const uint16_t*)q, (const uint16_t*)kc,
                                   (const uint16_t*)vc, kv_lens, max_len, (uint16_t*)o, tab.f32, B,
                                   Hq, Hkv, w_pre, w0, (float*)ws, s, ev0, ev1, block_table,
                                   max_pages, n_pages, page_shift, freq ? og : nullptr);
  if (e != hipSuccess) return hip_fail(e, "decode launch");
  return ok();
}

}  // namespace

extern "C" {

const char* jl_status_string(int status) {
  switch (status) {
    case JL_OK: return "JL_OK";
    case JL_ERR_INVALID_ARG: return "JL_ERR_INVALID_ARG";
    case JL_ERR_UNSUPPORTED: return "JL_ERR_UNSUPPORTED";
    case JL_ERR_WORKSPACE: return "JL_ERR_WORKSPACE";
    case JL_ERR_HIP: return "JL_ERR_HIP";
    default: return "JL_ERR_UNKNOWN";
  }
}

const char* jl_last_error(void) { return t_detail.c_str(); }

int jl_version(void) { return 100; }

int64_t jl_group_size(int64_t L, int64_t w_pretrained) {
  if (L < 1 || w_pretrained < 1) return -1;
  if (L <= w_pretrained) return 1;
  return (L + w_pretrained - 1) / w_pretrained;
}

int jl_bifocal_prefill(const void* q, const void* k, const void* v, void* o, float* lse, int B,
                       int Hq, int Hkv, int L, int head_dim, double rope_theta, int w_pretrained,
                       int w_local, void* stream) {
  return prefill_common(true, q, k, v, o, lse, B, Hq, Hkv, L, head_dim, rope_theta, w_pretrained,
                        w_local, stream);
}

int jl_rope_attention(const void* q, const void* k, const void* v, void* o, float* lse, int B,
                      int Hq, int Hkv, int L, int head_dim, double rope_theta, void* stream) {
  return prefill_common(false, q, k, v, o, lse, B, Hq, Hkv, L, head_dim, rope_theta, 1, 0,
                        stream);
}

int jl_bifocal_prefill_map(const void* q, const void* k, const void* v, void* o, float* lse,
                           int B, int Hq, int Hkv, int L, int head_dim, double rope_theta,
                           int w_pretrained, int w_local, int remote_map, void* stream) {
  return prefill_common(true, q, k, v, o, lse, B, Hq, Hkv, L, head_dim, rope_theta, w_pretrained,
                        w_local, stream, false, nullptr, 0, remote_map);
}

static int prefill_chunk(bool bifocal, const void* q, const void* k_cache, const void* v_cache,
                         void* o, float* lse, int B, int Hq, int Hkv, int q_start, int n_queries,
                         int max_len, int head_dim, double theta, int w_pre, int w0,
                         void* stream) {
  if (q_start < 0) return fail(JL_ERR_INVALID_ARG, "q_start must be >= 0 (got %d)", q_start);
  if (n_queries < 1) return fail(JL_ERR_INVALID_ARG, "n_queries must be >= 1 (got %d)", n_queries);
  if ((long long)q_start + n_queries > max_len)
    return fail(JL_ERR_INVALID_ARG, "q_start + n_queries (%lld) exceeds max_len (%d)",
                (long long)q_start + n_queries, max_len);
  return prefill_common(bifocal, q, k_cache, v_cache, o, lse, B, Hq, Hkv, q_start + n_queries,
                        head_dim, theta, w_pre, w0, stream, false, nullptr, 0, JL_REMOTE_ALIAS,
                        q_start, n_queries, max_len);
}

// A chunk over paged pools: the same call with key k of sequence b in page
// block_table[b][k / page_size].  Pages hold whole 64-key tiles, and the
// attention kernel keeps one sequence's page list in LDS.
static int prefill_chunk_paged(bool bifocal, const void* q, const void* k_pages,
                               const void* v_pages, const int32_t* block_table, int max_pages,
                               int page_size, int n_pages, void* o, float* lse, int B, int Hq,
                               int Hkv, int q_start, int n_queries, int head_dim, double theta,
                               int w_pre, int w0, void* stream) {
  if (!aligned4(block_table))
    return fail(JL_ERR_INVALID_ARG, "block_table must be non-null and 4-byte aligned");
  if (page_size < 1 || page_size > (1 << 20) || (page_size & (page_size - 1)) != 0)
    return fail(JL_ERR_INVALID_ARG, "page_size must be a power of two in [64, 2^20] (got %d)",
                page_size);
  if (page_size < kPagedPrefillMinPage)
    return fail(JL_ERR_UNSUPPORTED, "paged prefill needs page_size >= %d (got %d)",
                kPagedPrefillMinPage, page_size);
  if (max_pages < 1 || n_pages < 1)
    return fail(JL_ERR_INVALID_ARG, "max_pages and n_pages must be >= 1 (got %d, %d)", max_pages,
                n_pages);
  if (q_start < 0) return fail(JL_ERR_INVALID_ARG, "q_start must be >= 0 (got %d)", q_start);
  if (n_queries < 1) return fail(JL_ERR_INVALID_ARG, "n_queries must be >= 1 (got %d)", n_queries);
  const long long L = (long long)q_start + n_queries;
  if (L > (long long)max_pages * page_size)
    return fail(JL_ERR_INVALID_ARG, "q_start + n_queries (%lld) exceeds max_pages * page_size",
                L);
  if (L > 0x7fffffffLL) return fail(JL_ERR_INVALID_ARG, "q_start + n_queries too large");
  const long long pages = (L + page_size - 1) / page_size;
  if (pages > kPagedPrefillMaxPages)
    return fail(JL_ERR_UNSUPPORTED, "paged prefill reads %lld pages per sequence (at most %d)",
                pages, kPagedPrefillMaxPages);
  int page_shift = 0;
  while ((1 << page_shift) < page_size) ++page_shift;
  return prefill_common(bifocal, q, k_pages, v_pages, o, lse, B, Hq, Hkv, (int)L, head_dim,
                        theta, w_pre, w0, stream, false, nullptr, 0, JL_REMOTE_ALIAS, q_start,
                        n_queries, (int)L, block_table, max_pages, page_shift, n_pages);
}

int jl_bifocal_prefill_chunk_paged(const void* q, const void* k_pages, const void* v_pages,
                                   const int32_t* block_table, int max_pages, int page_size,
                                   int n_pages, void* o, float* lse, int B, int Hq, int Hkv,
                                   int q_start, int n_queries, int head_dim, double rope_theta,
                                   int w_pretrained, int w_local, void* stream) {
  return prefill_chunk_paged(true, q, k_pages, v_pages, block_table, max_pages, page_size,
                             n_pages, o, lse, B, Hq, Hkv, q_start, n_queries, head_dim,
                             rope_theta, w_pretrained, w_local, stream);
}

int jl_rope_attention_chunk_paged(const void* q, const void* k_pages, const void* v_pages,
                                  const int32_t* block_table, int max_pages, int page_size,
                                  int n_pages, void* o, float* lse, int B, int Hq, int Hkv,
                                  int q_start, int n_queries, int head_dim, double rope_theta,
                                  void* stream) {
  return prefill_chunk_paged(false, q, k_pages, v_pages, block_table, max_pages, page_size,
                             n_pages, o, lse, B, Hq, Hkv, q_start, n_queries, head_dim,
                             rope_theta, 1, 0, stream);
}

int jl_bifocal_prefill_chunk(const void* q, const void* k_cache, const void* v_cache, void* o,
                             float* lse, int B, int Hq, int Hkv, int q_start, int n_queries,
                             int max_len, int head_dim, double rope_theta, int w_pretrained,
                             int w_local, void* stream) {
  return prefill_chunk(true, q, k_cache, v_cache, o, lse, B, Hq, Hkv, q_start, n_queries, max_len,
                       head_dim, rope_theta, w_pretrained, w_local, stream);
}

int jl_rope_attention_chunk(const void* q, const void* k_cache, const void* v_cache, void* o,
                            float* lse, int B, int Hq, int Hkv, int q_start, int n_queries,
                            int max_len, int head_dim, double rope_theta, void* stream) {
  return prefill_chunk(false, q, k_cache, v_cache, o, lse, B, Hq, Hkv, q_start, n_queries,
                       max_len, head_dim, rope_theta, 1, 0, stream);
}

int jl_bifocal_prefill_varlen(const void* q, const void* k, const void* v, void* o, float* lse,
                              const int32_t* cu_seqlens, int B, int total_tokens, int max_seqlen,
                              int Hq, int Hkv, int head_dim, double rope_theta, int w_pretrained,
                              int w_local, void* stream) {
  return prefill_varlen(true, q, k, v, o, lse, cu_seqlens, B, total_tokens, max_seqlen, Hq, Hkv,
                        head_dim, rope_theta, w_pretrained, w_local, stream);
}

int jl_bifocal_prefill_varlen_map(const void* q, const void* k, const void* v, void* o,
                                  float* lse, const int32_t* cu_seqlens, int B, int total_tokens,
                                  int max_seqlen, int Hq, int Hkv, int head_dim, double rope_theta,
                                  int w_pretrained, int w_local, int remote_map, void* stream) {
  return prefill_varlen(true, q, k, v, o, lse, cu_seqlens, B, total_tokens, max_seqlen, Hq, Hkv,
                        head_dim, rope_theta, w_pretrained, w_local, stream, remote_map);
}

int jl_rope_attention_varlen(const void* q, const void* k, const void* v, void* o, float* lse,
                             const int32_t* cu_seqlens, int B, int total_tokens, int max_seqlen,
                             int Hq, int Hkv, int head_dim, double rope_theta, void* stream) {
  return prefill_varlen(false, q, k, v, o, lse, cu_seqlens, B, total_tokens, max_seqlen, Hq, Hkv,
                        head_dim, rope_theta, 1, 0, stream);
}

size_t jl_prefill_literal_workspace_bytes(int B, int Hq, int Hkv, int L, int head_dim) {
  if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || L < 1 || head_dim != kHeadDim) return 0;
  return jl::literal_workspace_bytes(B, Hq, Hkv, L);
}

int jl_bifocal_prefill_literal(const void* q, const void* k, const void* v, void* o, float* lse,
                               int B, int Hq, int Hkv, int L, int head_dim, double rope_theta,
                               int w_pretrained, int w_local, void* workspace,
                               size_t workspace_bytes, void* stream) {
  return prefill_common(true, q, k, v, o, lse, B, Hq, Hkv, L, head_dim, rope_theta, w_pretrained,
                        w_local, stream, true, workspace, workspace_bytes);
}

size_t jl_decode_map_workspace_bytes(int B, int Hq, int Hkv, int max_len, int head_dim,
                                     int remote_map) {
  if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || max_len < 1 || head_dim != kHeadDim) return 0;
  if (remote_map != JL_REMOTE_ALIAS && remote_map != JL_REMOTE_FREQ) return 0;
  return jl::decode_map_workspace_bytes(B, Hq, Hkv, max_len, remote_map == JL_REMOTE_FREQ);
}

int jl_bifocal_decode_map(const void* q, const void* k_cache, const void* v_cache,
                          const int32_t* kv_lens, int max_len, void* o, int B, int Hq, int Hkv,
                          int head_dim, double rope_theta, int w_pretrained, int w_local,
                          int remote_map, void* workspace, size_t workspace_bytes, void* stream) {
  return decode_common(true, q, k_cache, v_cache, kv_lens, max_len, o, B, Hq, Hkv, head_dim,
                       rope_theta, w_pretrained, w_local, workspace, workspace_bytes, stream,
                       nullptr, 0, 0, 0, remote_map);
}

size_t jl_decode_workspace_bytes(int B, int Hq, int Hkv, int max_len, int head_dim) {
  if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || max_len < 1 || head_dim != kHeadDim) return 0;
  return jl::decode_workspace_bytes(B, Hq, Hkv, max_len);
}

int jl_bifocal_decode(const void* q, const void* k_cache, const void* v_cache,
                      const int32_t* kv_lens, int max_len, void* o, int B, int Hq, int Hkv,
                      int head_dim, double rope_theta, int w_pretrained, int w_local,
                      void* workspace, size_t workspace_bytes, void* stream) {
  return decode_common(true, q, k_cache, v_cache, kv_lens, max_len, o, B, Hq, Hkv, head_dim,
                       rope_theta, w_pretrained, w_local, workspace, workspace_bytes, stream);
}

int jl_bifocal_decode_noalloc(const void* q, const void* k_cache, const void* v_cache,
                              const int32_t* kv_lens, int max_len, void* o, int B, int Hq,
                              int Hkv, int head_dim, double rope_theta, int w_pretrained,
                              int w_local, void* stream) {
  return decode_common(true, q, k_cache, v_cache, kv_lens, max_len, o, B, Hq, Hkv, head_dim,
                       rope_theta, w_pretrained, w_local, nullptr, 0, stream, nullptr, 0, 0, 0,
                       JL_REMOTE_ALIAS, true);
}

int jl_rope_attention_decode(const void* q, const void* k_cache, const void* v_cache,
                             const int32_t* kv_lens, int max_len, void* o, int B, int Hq,
                             int Hkv, int head_dim, double rope_theta, void* workspace,
                             size_t workspace_bytes, void* stream) {
  return decode_common(false, q, k_cache, v_cache, kv_lens, max_len, o, B, Hq, Hkv, head_dim,
                       rope_theta, 1, 0, workspace, workspace_bytes, stream);
}

int jl_bifocal_decode_paged(const void* q, const void* k_pages, const void* v_pages,
                            const int32_t* block_table, int max_pages, int page_size, int n_pages,
                            const int32_t* kv_lens, void* o, int B, int Hq, int Hkv,
                            int head_dim, double rope_theta, int w_pretrained, int w_local,
                            void* workspace, size_t workspace_bytes, void* stream) {
  if (block_table == nullptr) return fail(JL_ERR_INVALID_ARG, "block_table must be non-null");
  return decode_common(true, q, k_pages, v_pages, kv_lens, 0, o, B, Hq, Hkv, head_dim,
                       rope_theta, w_pretrained, w_local, workspace, workspace_bytes, stream,
                       block_table, max_pages, page_size, n_pages);
}

int jl_bifocal_decode_paged_map(const void* q, const void* k_pages, const void* v_pages,
                                const int32_t* block_table, int max_pages, int page_size,
                                int n_pages, const int32_t* kv_lens, void* o, int B, int Hq,
                                int Hkv, int head_dim, double rope_theta, int w_pretrained,
                                int w_local, int remote_map, void* workspace,
                                size_t workspace_bytes, void* stream) {
  if (block_table == nullptr) return fail(JL_ERR_INVALID_ARG, "block_table must be non-null");
  return decode_common(true, q, k_pages, v_pages, kv_lens, 0, o, B, Hq, Hkv, head_dim,
                       rope_theta, w_pretrained, w_local, workspace, workspace_bytes, stream,
                       block_table, max_pages, page_size, n_pages, remote_map);
}

int jl_rope_attention_decode_paged(const void* q, const void* k_pages, const void* v_pages,
                                   const int32_t* block_table, int max_pages, int page_size,
                                   int n_pages, const int32_t* kv_lens, void* o, int B, int Hq,
                                   int Hkv, int head_dim, double rope_theta, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  if (block_table == nullptr) return fail(JL_ERR_INVALID_ARG, "block_table must be non-null");
  return decode_common(false, q, k_pages, v_pages, kv_lens, 0, o, B, Hq, Hkv, head_dim,
                       rope_theta, 1, 0, workspace, workspace_bytes, stream, block_table,
                       max_pages, page_size, n_pages);
}

int jl_debug_schedule(const int32_t* lengths, int n_lengths, const int32_t* positions,
                      int n_positions, int w_pretrained, int32_t* group_out, int32_t* remote_out,
                      int32_t* offset_out, void* stream) {
  if (n_lengths < 0 || n_positions < 0)
    return fail(JL_ERR_INVALID_ARG, "counts must be >= 0");
  if (w_pretrained < 1) return fail(JL_ERR_INVALID_ARG, "w_pretrained must be >= 1");
  if (n_lengths > 0 && n_positions > 0) {
    if (!aligned4(lengths) || !aligned4(positions) || !aligned4(group_out) ||
        !aligned4(remote_out) || !aligned4(offset_out))
      return fail(JL_ERR_INVALID_ARG, "null or misaligned pointer");
    if ((long long)n_lengths * n_positions > 0x7fffffffLL)
      return fail(JL_ERR_INVALID_ARG, "problem too large");
  }
  hipError_t e = jl::launch_debug_schedule(lengths, n_lengths, positions, n_positions,
                                           w_pretrained, group_out, remote_out, offset_out,
                                           reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "debug schedule launch");
  return ok();
}

int jl_debug_prefill_tiles(int L, int Hq, int Hkv, int w_local, int8_t* classes_out,
                           int64_t classes_len, int* block_q, int* block_k, int* n_qblocks,
                           int* n_ktiles, void* stream) {
  if (L < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || w_local < 0)
    return fail(JL_ERR_INVALID_ARG, "invalid L, Hq, Hkv or w_local");
  if (jl::prefill_rows_per_block() % (Hq / Hkv) != 0)
    return fail(JL_ERR_UNSUPPORTED, "GQA group must divide the block's rows");
  if (!block_q || !block_k || !n_qblocks || !n_ktiles)
    return fail(JL_ERR_INVALID_ARG, "null geometry pointer");
  const int BQ = jl::prefill_block_q(Hq / Hkv), BK = jl::prefill_block_k();
  const int nqb = (L + BQ - 1) / BQ, nkt = (L + BK - 1) / BK;
  *block_q = BQ;
  *block_k = BK;
  *n_qblocks = nqb;
  *n_ktiles = nkt;
  if (classes_out == nullptr || classes_len < (int64_t)nqb * nkt)
    return fail(JL_ERR_INVALID_ARG, "classes_out needs %lld elements",
                (long long)nqb * nkt);
  hipError_t e = jl::launch_debug_tiles(L, BQ, BK, w_local, nqb, nkt, classes_out,
                                        reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "debug tiles launch");
  return ok();
}

int jl_debug_kernel_events(int which, void* start, void* stop) {
  if (which != 0 && which != 1) return fail(JL_ERR_INVALID_ARG, "which must be 0 or 1");
  if ((start == nullptr) != (stop == nullptr))
    return fail(JL_ERR_INVALID_ARG, "start and stop must both be set or both be NULL");
  std::lock_guard<std::mutex> lock(g_ev_mu);
  g_events[which][0] = reinterpret_cast<hipEvent_t>(start);
  g_events[which][1] = reinterpret_cast<hipEvent_t>(stop);
  return ok();
}

double jl_debug_prefill_rescale_log2(double log2_bound) {
  if (!(log2_bound >= 1.0 && log2_bound <= 100.0)) return g_rescale_log2.load();
  return g_rescale_log2.exchange(log2_bound);
}

void jl_release_caches(void) {
  std::lock_guard<std::mutex> lock(g_mu);
  int cur = 0;
  const bool have_cur = hipGetDevice(&cur) == hipSuccess;
  for (auto& t : g_tables) {
    if (hipSetDevice(t.device) == hipSuccess) (void)hipFree(t.ptr);
  }
  for (auto& r : g_retired) {
    if (hipSetDevice(r.first) == hipSuccess) (void)hipFree(r.second);
  }
  for (auto& t : g_freq_tables) {
    if (hipSetDevice(t.device) == hipSuccess) (void)hipFree(t.ptr);
  }
  for (auto& sc : g_scratch) {
    if (hipSetDevice(sc.device) == hipSuccess) {
      (void)hipStreamSynchronize(sc.stream);
      (void)hipFree(sc.ptr);
    }
  }
  g_tables.clear();
  g_freq_tables.clear();
  g_retired.clear();
  g_scratch.clear();
  if (have_cur) (void)hipSetDevice(cur);
}

}  // extern "C"
