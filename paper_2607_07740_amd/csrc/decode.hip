// decode.hip -- single-query bifocal-RoPE decode on a raw KV cache, gfx950.
//
// Jet-Long (arXiv 2607.07740), Sec. 3.2: the cache keeps keys in their base
// coordinates and is never rewritten when G changes; the remote view of a key
// is formed on the fly by rotating it to f(k) (the correction rotation of
// Eqs. (5)-(6), applied here to raw keys as R(f(k)) x_k = R(Delta k) R(k) x_k).
// The query of sequence b sits at q = kv_len[b] - 1 and G follows from
// L = kv_len[b] (Eq. (2)), computed on the device, so one launch serves a
// ragged batch whose sequences have different G.
//
// Split-K: workgroup (b, group of up to 4 kv heads, split) streams every
// ns_b-th 16-key step of sequence b, two waves per kv head; ns_b follows the
// sequence's length (split_work), so a ragged batch keeps every CU busy for
// about the same time.  The Sec. 4.5 frequency map replaces the remote
// rotation by one at unchanged positions with rescaled frequencies.  The g query
// heads of a kv head are rotated twice (base and remote) and placed in the 16
// columns of a v_mfma_f32_16x16x32_bf16 B operand: columns 0..7 hold
// the base-rotated heads, 8..15 the remote-rotated ones.  Each key is rotated
// once, to the view its distance selects (Eq. (1)), and scored against both
// column groups; a column keeps only keys of its own view, so every column is
// the partial softmax state (m, l, O) of one (head, view) pair: the local
// window state and the remote-only state of Sec. 3.3.  Each split merges its
// head's two view states with the max-shifted, linear-space rule of Eq. (7)
// in fp32, and the reduce kernel merges the splits' states the same way.
#include <mutex>

#include "jl_device.h"

namespace jl {

constexpr int kDecHeads = 4;  // kv heads per workgroup
constexpr int kDecWaves = 8;  // two waves per head: one takes the even steps, one the odd
constexpr int kDecThreads = 64 * kDecWaves;
constexpr int kDecTile = 16;  // keys per step
constexpr int kDecBufs = 4;   // LDS buffers: the two steps in use and the next two in flight
constexpr int kDecImgBytes = kDecTile * kDecHeads * kHeadDim * 2;  // K or V of one step: 16 KB
constexpr int kDecBufBytes = 2 * kDecImgBytes + 1024;  // K, V and the step's two query cos/sin rows
constexpr int kDecOffTab = kDecBufs * kDecBufBytes;
constexpr int kDecTabRow = kHalf * 8 + 16;  // one offset row: 64 (cos, sin) pairs + 16 B pad
constexpr int kDecOffTab2 = kDecOffTab + kDecTile * kDecTabRow;    // + 16 offset rows (base)
constexpr int kDecOffDummy = kDecOffTab2 + kDecTile * kDecTabRow;  // + 16 offset rows (freq map)
constexpr int kDecOffPages = kDecOffDummy + 1024;                  // + landing slot for padding copies
constexpr int kDecPageCap = 2048;  // paged caches: page indices of up to this many steps in LDS
constexpr int kDecSmem = kDecOffPages + kDecPageCap * 4;
constexpr int kDecCopies = 5;  // copies per step of wave 0: four K/V (padded to a fixed count) + rows
constexpr int kStateFloats = 132;  // m, l, the split count (int bits), pad, O[128]

struct DecodeArgs {
  const uint16_t* q;
  const uint16_t* kc;
  const uint16_t* vc;
  const int32_t* kv_lens;
  float* ws;
  const float2* table;
  int B, Hq, Hkv, g, max_len;  // max_len: most keys a sequence can hold
  // paged caches: kc, vc are pools [n_pages][page_size][Hkv][128] and key k of
  // sequence b sits in page block_table[b][k >> page_shift]; nullptr: dense
  // caches [B][max_len][Hkv][128]
  const int32_t* block_table;
  int max_pages, n_pages, page_shift;
  int chunk, n_split, n_hgroups;  // n_split: split slots per (b, kv-head group)
  int balanced;  // split counts from the actual lengths (B <= 64), else from max_len
  // frequency-interpolation remote map (Sec. 4.5): omega_i and the ramp
  // gamma_i of each frequency pair; every workgroup forms the cos/sin rows it
  // needs from them and its sequence's length
  double fomega[kHalf];
  double fgamma[kHalf];
  int n_target;  // balanced: workgroups of the grid (one wave of them fills the GPU)
  int w_pre, w0;
  float q_scale;
};

__device__ inline int clamp_len(int n, int max_len) { return n < 1 ? 1 : (n > max_len ? max_len : n); }

__device__ inline int wave_sum(int x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

__device__ inline int wave_max(int x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = max(x, __shfl_xor(x, o));
  return x;
}

// 16-key steps of sequence `lane` (0 for lanes past B)
__device__ inline int lane_steps(const DecodeArgs& a, int lane) {
  return lane < a.B ? (clamp_len(a.kv_lens[lane], a.max_len) + kDecTile - 1) / kDecTile : 0;
}

// Balanced splits of a ragged batch (one lane per sequence, s = its steps):
// every split takes at most u steps, u the smallest count for which the
// busy workgroups, n_hgroups * sum_b min(n_split, ceil(s_b / u)), fit the
// grid's n_target slots; the bisection starts from the bounds
//   ceil(total / S) <= u <= ceil(total / (S - B))   (S = n_target / n_hgroups)
// since sum_b ceil(s_b / u) lies between total / u and total / u + B.
__device__ inline int balanced_unit(const DecodeArgs& a, int s) {
  const int S = a.n_target / a.n_hgroups;  // >= B
  const int smax = wave_max(s);
  if (a.B == 1) return max(1, (smax + S - 1) / S);
  const int total = wave_sum(s);
  int lo = max(1, (total + S - 1) / S);
  int hi = S > a.B ? min(smax, (total + S - a.B - 1) / (S - a.B)) : smax;
  lo = min(lo, hi);
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    const int c = wave_sum(s > 0 ? min(a.n_split, (s + mid - 1) / mid) : 0);
    if (c <= S) hi = mid; else lo = mid + 1;
  }
  return lo;
}

// What workgroup bid does: sequence b, kv-head group, split `split` of ns
// (ns == 0: nothing, the workgroup exits).  Balanced grids list, per
// sequence, its ns_b * n_hgroups workgroups one after another.
struct SplitWork {
  int b, hgroup, split, ns;
};

__device__ inline SplitWork split_work(const DecodeArgs& a, int bid) {
  SplitWork w;
  if (!a.balanced) {
    w.split = bid % a.n_split;
    const int t0 = bid / a.n_split;
    w.hgroup = t0 % a.n_hgroups;
    w.b = t0 / a.n_hgroups;
    const int s_all = (clamp_len(a.kv_lens[w.b], a.max_len) + kDecTile - 1) / kDecTile;
    w.ns = min(a.n_split, s_all);
    if (w.split >= w.ns) w.ns = 0;
    return w;
  }
  const int lane = threadIdx.x & 63;
  const int s = lane_steps(a, lane);
  const int u = balanced_unit(a, s);
  const int ns = s > 0 ? min(a.n_split, (s + u - 1) / u) : 0;
  int incl = ns * a.n_hgroups;  // inclusive scan over the sequences
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int x = __shfl_up(incl, o);
    if (lane >= o) incl += x;
  }
  const int b = __popcll(__ballot(lane < a.B && incl <= bid));
  w.b = min(b, a.B - 1);
  const int incl_b = __shfl(incl, w.b);
  const int ns_b = __shfl(ns, w.b);
  const int r = bid - (incl_b - ns_b * a.n_hgroups);
  w.ns = b < a.B ? ns_b : 0;
  w.hgroup = w.ns > 0 ? r / ns_b : 0;
  w.split = w.ns > 0 ? r - w.hgroup * ns_b : 0;
  w.b = __builtin_amdgcn_readfirstlane(w.b);
  w.ns = __builtin_amdgcn_readfirstlane(w.ns);
  w.hgroup = __builtin_amdgcn_readfirstlane(w.hgroup);
  w.split = __builtin_amdgcn_readfirstlane(w.split);
  return w;
}

// Rotate 8 (d, d + 64) pairs given in fp32 by the (cos, sin) pairs c4[0..3]
// (frequencies d..d+7).
__device__ inline void rotate8f(const float* lo, const float* hi, const float4* c4, bf16x8& olo,
                                bf16x8& ohi) {
  float ylo[8], yhi[8];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    float4 w = c4[t];
    int j = 2 * t;
    ylo[j] = lo[j] * w.x - hi[j] * w.y;
    yhi[j] = hi[j] * w.x + lo[j] * w.y;
    ylo[j + 1] = lo[j + 1] * w.z - hi[j + 1] * w.w;
    yhi[j + 1] = hi[j + 1] * w.z + lo[j + 1] * w.w;
  }
  olo = pack8(ylo);
  ohi = pack8(yhi);
}

// Rotate an 8-element pair of slices (d, d + 64) by the (cos, sin) pairs c4[0..3]
// (frequencies d..d+7), optional scale.
__device__ inline void rotate8(const u32x4 rlo, const u32x4 rhi, const float4* c4, float scale,
                               bf16x8& olo, bf16x8& ohi) {
  float lo[8], hi[8], ylo[8], yhi[8];
  unpack8(rlo, lo);
  unpack8(rhi, hi);
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    float4 w = c4[t];
    int j = 2 * t;
    ylo[j] = (lo[j] * w.x - hi[j] * w.y) * scale;
    yhi[j] = (hi[j] * w.x + lo[j] * w.y) * scale;
    ylo[j + 1] = (lo[j + 1] * w.z - hi[j + 1] * w.w) * scale;
    yhi[j + 1] = (hi[j + 1] * w.z + lo[j + 1] * w.w) * scale;
  }
  olo = pack8(ylo);
  ohi = pack8(yhi);
}

__device__ inline f32x4 mfma16k16(bf16x4 a, bf16x4 b, f32x4 c) {
  typedef short i16x4v __attribute__((ext_vector_type(4)));
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4v, a),
                                                   __builtin_bit_cast(i16x4v, b), c, 0, 0, 0);
}

// Split-K workgroup (b, group of up to 4 kv heads, split): split s takes the
// 16-key steps s, s + n_split, s + 2 n_split, ... of the sequence, so at any
// moment all workgroups stream one narrow window of the cache.  Every 16-key
// step copies the keys' contiguous head slices (K and V, one key's heads are
// adjacent in the cache) straight into LDS.  Waves w and w + 4 serve kv head
// 4 * group + w on the even and the odd steps, so two waves share each SIMD
// and hide each other's latency; their partial states are merged at the end.
// Four buffers hold the two steps being computed and the next two in flight.
//
// Rotation by tile offset: with k0 the step's first key, a key at k0 + t is
// rotated by t only, R(t) x_k (base view) or by f(k0 + t) - f(k0) (remote
// view), from 16 cos/sin rows kept in LDS, and the query columns are rotated
// by q - k0 or f(q) - f(k0) instead: <R(a) x_q, R(b) x_k> = <R(a - c) x_q,
// R(b - c) x_k> for any c (rotations compose additively, Sec. 3.2 Eq. (6)).
// So no per-key cos/sin row is fetched from memory; the step's two query rows
// arrive with its copies.
//
// LDS layouts (16-byte slots inside one head's 256-byte row of a key t):
//   K: slot s holds chunk s ^ t          (16 keys read at one d: 16 bank groups)
//   V: slot s holds chunk s ^ 2 (t & 7)  (8 keys x 32 B of a transposing read)
//   offset table row r (512 B + 16 B pad, so the 16 rows start 4 banks
//   apart): slot s holds frequencies 2 s, 2 s + 1
// RMODE: 0 the vanilla kernel, 1 bifocal with the Eq. (3) map, 2 bifocal with
// the frequency map (remote rotations at unchanged positions by omega').
// The Sec. 4.5 map of a sequence of n keys: s = max(1, n / w_pretrained) and
// omega'_i = (1 - gamma_i) omega_i / s + gamma_i omega_i (freq_map_omega);
// the (cos, sin) of pos * omega'_i (freq_map_cs), with the angle formed and
// reduced modulo 2 pi in fp64 (exact to ~1e-11 rad at 1.3e5 rad) and its sine
// and cosine taken in fp32, within an ulp or two of the fp64 result rounded
// to fp32.
__device__ inline double freq_map_omega(const DecodeArgs& a, int n, int i) {
#pragma clang fp contract(off)
  const double om = a.fomega[i];
  const double sc = fmax(1.0, (double)n / (double)a.w_pre);
  return (1.0 - a.fgamma[i]) * om / sc + a.fgamma[i] * om;
}
__device__ inline float2 freq_map_cs(double omf, int pos) {
#pragma clang fp contract(off)
  const double two_pi = 6.283185307179586476925286766559;
  double ang = (double)pos * omf;
  ang -= two_pi * rint(ang * (1.0 / two_pi));
  float sn, cs;
  sincosf((float)ang, &sn, &cs);
  return make_float2(cs, sn);
}

template <int RMODE>
__global__ __launch_bounds__(kDecThreads, 1) void decode_split_kernel(DecodeArgs a) {
  constexpr bool BIFOCAL = RMODE != 0;
  constexpr bool FREQ = RMODE == 2;
  __shared__ __attribute__((aligned(1024))) unsigned char smem[kDecSmem];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int hw = wave & (kDecHeads - 1);  // head slot
  const int par = wave / kDecHeads;       // step parity
  const int i16 = lane & 15;
  const int g4 = lane >> 4;

  const SplitWork sw = split_work(a, blockIdx.x);
  if (sw.ns == 0) return;  // whole workgroup, before any barrier
  const int split = sw.split, hgroup = sw.hgroup, b = sw.b, ns = sw.ns;
  const int h0 = hgroup * kDecHeads;
  const int Hg = min(kDecHeads, a.Hkv - h0);  // heads in this group
  const int kvh = h0 + hw;
  const bool head_on = hw < Hg;
  const int kv_len = clamp_len(a.kv_lens[b], a.max_len);
  // this split's steps: global 16-key steps split, split + ns, ... below
  // kv_len, so at any moment all splits read neighbouring parts of the cache
  const int s_all = (kv_len + kDecTile - 1) / kDecTile;
  const int c1 = kv_len;
  const int kstride = ns * kDecTile;
  const int c0 = split * kDecTile;
  const int G = BIFOCAL ? group_size(kv_len, a.w_pre) : 1;
  const FastDiv gdiv = make_fastdiv((uint32_t)G);
  const int qpos = kv_len - 1;
  const int fq = BIFOCAL ? remote_pos(qpos, gdiv) : qpos;
  // the frequency map's omega'_i of this lane's frequency (wave 0 forms the
  // step rows, lane i taking frequency i)
  const double omf_lane = FREQ ? freq_map_omega(a, kv_len, lane) : 0.0;
  const int n_steps = (s_all - split + ns - 1) / ns;
  const int n_iter = (n_steps + 1) / 2;

  // ---- copies: a step's K image is 16 keys x Hg heads x 256 B = 4 Hg chunks
  // of 1 KB, V likewise; chunk n < 4 Hg is K, n < 8 Hg is V.  Wave w takes
  // chunks w + 8 i, i < 4; past 8 Hg it copies into a landing slot nobody
  // reads, so every wave has the same number of copies per step.  Lane ->
  // LDS slot 16 * lane of its chunk; it fetches the global chunk that slot
  // holds (keys past the chunk read the chunk's last key).
  const uint32_t row_bytes = (uint32_t)Hg * 256;
  const uint32_t smem_base = lds_addr(smem);
  const unsigned char* kbase = (const unsigned char*)(a.kc + (size_t)h0 * kHeadDim);
  const unsigned char* vbase = (const unsigned char*)(a.vc + (size_t)h0 * kHeadDim);
  const uint32_t kv_row_bytes = (uint32_t)a.Hkv * 256;
  // cache row of step jb's first key: a step's 16 keys are consecutive rows
  // (pages hold a multiple of 16 keys).  The page index is read first
  // (step_page) and turned into a row where the copies are issued (step_row),
  // so the table read overlaps the compute in between; page indices are
  // clamped to the pool.
  int32_t* pages_lds = (int32_t*)(smem + kDecOffPages);
  const bool pages_in_lds = a.block_table != nullptr && n_steps <= kDecPageCap;
  auto step_page = [&](int jb) {
    if (a.block_table == nullptr) return 0;
    if (pages_in_lds) return (int)pages_lds[min(jb, n_steps - 1)];
    const int k0 = c0 + min(jb, n_steps - 1) * kstride;
    // the table is read-only for the kernel: read it through the constant
    // address space, so the load is a scalar one and its wait does not
    // drain the outstanding copies
    typedef __attribute__((address_space(4))) const int32_t const_i32;
    const const_i32* bt = (const const_i32*)a.block_table;
    return (int)bt[(size_t)b * a.max_pages + (k0 >> a.page_shift)];
  };
  auto step_row = [&](int jb, int pg) {
    const int k0 = c0 + min(jb, n_steps - 1) * kstride;
    if (a.block_table == nullptr) return (size_t)b * a.max_len + k0;
    pg = min(max(pg, 0), a.n_pages - 1);
    return ((size_t)pg << a.page_shift) + (k0 & ((1 << a.page_shift) - 1));
  };
  // per copy i of this lane: the key row t it serves and the byte offset of its
  // chunk inside that key's slice of the cache (the same for every step)
  uint32_t cp_t[kDecCopies - 1], cp_off[kDecCopies - 1];
#pragma unroll
  for (int i = 0; i < kDecCopies - 1; ++i) {
    const int n = wave + kDecWaves * i;
    const bool is_v = n >= 4 * Hg;
    const bool real = n < 8 * Hg;
    const uint32_t o = (real ? (is_v ? n - 4 * Hg : n) : 0) * 1024 + 16 * lane;
    const uint32_t t = o / row_bytes;
    const uint32_t rem = o - t * row_bytes;
    const uint32_t h = rem >> 8, slot = (rem & 255) >> 4;
    cp_t[i] = t;
    cp_off[i] = h * 256 + 16 * (slot ^ (is_v ? 2 * (t & 7) : t));
  }
  uint32_t cp_full[kDecCopies - 1];  // byte offsets inside a step with 16 valid keys
#pragma unroll
  for (int i = 0; i < kDecCopies - 1; ++i) cp_full[i] = cp_t[i] * kv_row_bytes + cp_off[i];
  auto issue = [&](int jb, size_t row0) {
    const int k0 = c0 + min(jb, n_steps - 1) * kstride;
    const uint32_t buf = smem_base + (jb % kDecBufs) * kDecBufBytes;
    const unsigned char* kstep = kbase + row0 * kv_row_bytes;
    const unsigned char* vstep = vbase + row0 * kv_row_bytes;
    if (wave == 0) {
      // the cos/sin rows that rotate the query columns for this step: q - k0
      // (lanes 0..31) and f(q) - f(k0) (lanes 32..63) of the table, or the
      // step's row pair of the frequency map; one copy, by wave 0 alone (the
      // other waves wait for one copy fewer per step)
      const uint32_t dst = buf + 2 * kDecImgBytes;
      if (FREQ) {
        // the base row copied by lanes 0..31; the frequency map's row R'(q -
        // k0) formed here, lane i taking frequency i, and stored beside it
        if (lane < 32) dma16_s(a.table, (uint32_t)(qpos - k0) * 512 + 16 * lane, dst);
        const float2 cs = freq_map_cs(omf_lane, qpos - k0);
        *(float2*)(smem + (dst - smem_base) + 512 + 8 * lane) = cs;
      } else {
        const int fk0 = BIFOCAL ? remote_pos(k0, gdiv) : k0;
        const int row = lane < 32 ? qpos - k0 : fq - fk0;
        dma16_s(a.table, (uint32_t)row * 512 + 16 * (lane & 31), dst);
      }
    }
    // K and V are read exactly once per call: nontemporal.  A step whose 16
    // keys all lie below kv_len (every step but a sequence's last) takes the
    // precomputed offsets; the last one repeats its last key past kv_len.
    auto copy = [&](int i, uint32_t voff) __attribute__((always_inline)) {
      const int n = wave + kDecWaves * i;  // wave-uniform
      const bool is_v = n >= 4 * Hg;
      const bool real = n < 8 * Hg;
      const uint32_t dst = real ? buf + (is_v ? kDecImgBytes + (n - 4 * Hg) * 1024 : n * 1024)
                                : smem_base + kDecOffDummy;
      dma16_s_nt(is_v && real ? vstep : kstep, voff, dst);
    };
    if (k0 + kDecTile <= c1) {  // wave-uniform
#pragma unroll
      for (int i = 0; i < kDecCopies - 1; ++i) copy(i, cp_full[i]);
    } else {
#pragma unroll
      for (int i = 0; i < kDecCopies - 1; ++i)
        copy(i, (uint32_t)(min(k0 + (int)cp_t[i], c1 - 1) - k0) * kv_row_bytes + cp_off[i]);
    }
  };

  // ---- offset table: cos/sin of t * omega_i for t = 0..15 (table rows 0..15)
  {
    unsigned char* tab = smem + kDecOffTab;
    for (int i = threadIdx.x; i < kDecTile * 32; i += kDecThreads) {
      const int r = i >> 5, s = i & 31;
      *(float4*)(tab + r * kDecTabRow + 16 * s) = *(const float4*)(a.table + r * kHalf + 2 * s);
      if (FREQ) {
        // the frequency map's rows t omega'_i, t = 0..15
        const float2 c0 = freq_map_cs(freq_map_omega(a, kv_len, 2 * s), r),
                     c1 = freq_map_cs(freq_map_omega(a, kv_len, 2 * s + 1), r);
        *(float4*)(tab + (kDecOffTab2 - kDecOffTab) + r * kDecTabRow + 16 * s) =
            make_float4(c0.x, c0.y, c1.x, c1.y);
      }
    }
  }
  const unsigned char* tab = smem + kDecOffTab;

  // ---- query columns: col = (view, head) with view = col / 8; raw slices kept
  const int col = i16;
  const int view = col >> 3;
  const int hj = col & 7;
  const bool col_on = head_on && hj < a.g && (BIFOCAL || view == 0);
  // distances q - k this column keeps: [keep_lo, keep_lo + keep_n) as one
  // unsigned compare; base view 0 .. w0 (every causal key for the vanilla
  // kernel), remote view w0 + 1 .. INT_MAX (Eq. (1)), none for unused columns
  const int keep_lo = BIFOCAL && view == 1 ? (int)min((uint32_t)a.w0 + 1u, (uint32_t)INT_MAX) : 0;
  const uint32_t keep_n = !col_on ? 0u
                          : !BIFOCAL ? 0x80000000u
                          : view == 0 ? (uint32_t)a.w0 + 1u
                                      : (uint32_t)INT_MAX - (uint32_t)a.w0;
  // the raw query slices in fp32, scaled once (log2(e) / sqrt(d)): every
  // step rotates them by its own offset without unpacking or scaling again
  float qf[4][8];
  {
    const uint16_t* qrow =
        a.q + ((size_t)b * a.Hq + min(kvh, a.Hkv - 1) * a.g + min(hj, a.g - 1)) * kHeadDim;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      unpack8(load16(qrow + 32 * s + 8 * g4), qf[s]);
#pragma unroll
      for (int i = 0; i < 8; ++i) qf[s][i] *= a.q_scale;
    }
  }

  // paged caches: the page index of every step of this split, into LDS
  if (pages_in_lds) {
    for (int j = threadIdx.x; j < n_steps; j += kDecThreads) {
      const int k0 = c0 + j * kstride;
      pages_lds[j] = a.block_table[(size_t)b * a.max_pages + (k0 >> a.page_shift)];
    }
    __syncthreads();
  }

  // the plain loads above complete before the first copy is requested, so the
  // compiler's waits for them never hold back the copies
  wait_vmem();
  for (int jb = 0; jb < 4; ++jb) issue(jb, step_row(jb, step_page(jb)));

  f32x4 acc_o[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc_o[i] = f32x4{};
  float m_run = -INFINITY, l_run = 0.f;

  for (int it = 0; it < n_iter; ++it) {
    // cache rows of the steps copied at the end of this iteration, looked up
    // now so the block-table reads are long done by then
    const int page4 = step_page(2 * it + 4), page5 = step_page(2 * it + 5);
    // this wave's copies of steps 2it, 2it+1 (the next pair may fly): four
    // K/V copies per step, and in wave 0 the step's query cos/sin row too
    if (wave == 0)
      wait_vmem_n<2 * kDecCopies>();
    else
      wait_vmem_n<2 * (kDecCopies - 1)>();
    __syncthreads();  // everyone's copies (and the offset table)
    const int j = 2 * it + par;
    if (head_on && j < n_steps) {
      const int k0 = c0 + j * kstride;
      const unsigned char* sb = smem + (j % kDecBufs) * kDecBufBytes;
      const unsigned char* kb = sb + hw * 256;
      const unsigned char* vb = kb + kDecImgBytes;
      const int fk0 = BIFOCAL ? remote_pos(k0, gdiv) : k0;

      // query operand rotated by q - k0 (base columns) or f(q) - f(k0) (remote)
      bf16x8 qop[4];
      {
        const float4* c4 = (const float4*)(sb + 2 * kDecImgBytes + 512 * view);
#pragma unroll
        for (int s = 0; s < 2; ++s)
          rotate8f(qf[s], qf[s + 2], c4 + 16 * s + 4 * g4, qop[s], qop[s + 2]);
        if (!col_on) {
#pragma unroll
          for (int s = 0; s < 4; ++s) qop[s] = bf16x8{};
        }
      }

      // key t = i16 of this lane, rotated once, by its view's offset
      const int key = k0 + i16;
      // remote keys: offset f(k) - f(k0) in the base rows (Eq. (3)), or t in
      // the frequency map's rows
      int r = i16;
      if (BIFOCAL && qpos - key > a.w0)
        r = FREQ ? i16 + (kDecOffTab2 - kDecOffTab) / kDecTabRow : remote_pos(key, gdiv) - fk0;
      f32x4 sc = f32x4{};
      {
        u32x4 kr[4];
#pragma unroll
        for (int s = 0; s < 4; ++s)
          kr[s] = *(const u32x4*)(kb + i16 * row_bytes + 16 * ((4 * s + g4) ^ i16));
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          float4 cs[4];
#pragma unroll
          for (int u = 0; u < 4; ++u)
            cs[u] = *(const float4*)(tab + r * kDecTabRow + 16 * (16 * s + 4 * g4 + u));
          bf16x8 lo, hi;
          rotate8(kr[s], kr[s + 2], cs, 1.f, lo, hi);
          sc = mfma16(lo, qop[s], sc);
          sc = mfma16(hi, qop[s + 2], sc);
        }
      }

      // each column keeps only the keys of its own view (q - k in [lo, lo +
      // keep)); lane holds keys 4 g4 + i
      float sv[4];
      const uint32_t dbase = (uint32_t)(qpos - k0 - 4 * g4) - (uint32_t)keep_lo;
#pragma unroll
      for (int i = 0; i < 4; ++i) sv[i] = dbase - (uint32_t)i < keep_n ? sc[i] : -INFINITY;

      // online softmax per column (the 4 lanes i16, i16+16, i16+32, i16+48)
      float mt = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
      mt = fmaxf(mt, __shfl_xor(mt, 16));
      mt = fmaxf(mt, __shfl_xor(mt, 32));
      const float m_new = fmaxf(m_run, mt);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      // 1 unless the maximum moved (a column with no key of its view yet
      // keeps m = -inf and must not take the rescale branch every step)
      const float alpha = m_new == m_run ? 1.f : fast_exp2(m_run - m_use);
      f32x4 p;
#pragma unroll
      for (int i = 0; i < 4; ++i) p[i] = fast_exp2(sv[i] - m_use);
      l_run = l_run * alpha + (p[0] + p[1]) + (p[2] + p[3]);
      m_run = m_new;
      if (__ballot(alpha != 1.f) != 0) {  // most steps leave every column's maximum alone
#pragma unroll
        for (int db = 0; db < 8; ++db) acc_o[db] *= alpha;
      }
      // P^T operand of the k = 16 product: k index 4 g4 + i is key 4 g4 + i
      const bf16x4 pb = __builtin_convertvector(p, bf16x4);

      // O^T += V^T P^T; a transposing read gives lane i of group g4 the keys
      // 4 g4 .. 4 g4 + 3 at d = 16 db + i
#pragma unroll
      for (int db = 0; db < 8; ++db) {
        const int c = 2 * db + ((i16 & 3) >> 1);
        const int ta = 4 * g4 + (i16 >> 2);
        const i16x4 v =
            lds_read_tr4(vb + ta * row_bytes + 16 * (c ^ (2 * (ta & 7))) + 8 * (i16 & 1));
        acc_o[db] = mfma16k16(__builtin_bit_cast(bf16x4, v), pb, acc_o[db]);
      }
    }
    __syncthreads();  // steps 2it, 2it+1 consumed: their buffers take steps 2it+4, 2it+5
    issue(2 * it + 4, step_row(2 * it + 4, page4));
    issue(2 * it + 5, step_row(2 * it + 5, page5));
  }
  wait_vmem();  // copies requested past the last step
  __syncthreads();  // every buffer is free again

  // ---- merge the odd-step wave's state into the even-step wave's (max-shifted)
  {
    float* xs = (float*)smem + ((size_t)hw * 64 + lane) * 34;
    if (par == 1) {
      xs[0] = m_run;
      xs[1] = l_run;
#pragma unroll
      for (int db = 0; db < 8; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i) xs[2 + 4 * db + i] = acc_o[db][i];
    }
    __syncthreads();
    if (par == 1 || !head_on) return;
    const float m_b = xs[0];
    const float M = fmaxf(m_run, m_b);
    const float wa = M == -INFINITY ? 0.f : fast_exp2(m_run - M);
    const float wb = M == -INFINITY ? 0.f : fast_exp2(m_b - M);
    l_run = wa * l_run + wb * xs[1];
#pragma unroll
    for (int db = 0; db < 8; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc_o[db][i] = wa * acc_o[db][i] + wb * xs[2 + 4 * db + i];
    m_run = M;
  }

  // ---- one state per head: Eq. (7) over the local-window state (column hj)
  // and the remote-only state (column 8 + hj); the exclusion window is empty
  // because band keys never enter the remote view
  float l_tot = l_run + __shfl_xor(l_run, 16);
  l_tot += __shfl_xor(l_tot, 32);
  float m_own = m_run, l_own = l_tot;
  float W_own = 1.f, W_oth = 0.f;
  float m_oth = -INFINITY, l_oth = 0.f;
  if (BIFOCAL) {
    m_oth = __shfl_xor(m_run, 8);
    l_oth = __shfl_xor(l_tot, 8);
    const float M = fmaxf(m_own, m_oth);
    W_own = M == -INFINITY ? 0.f : fast_exp2(m_own - M);
    W_oth = M == -INFINITY ? 0.f : fast_exp2(m_oth - M);
    m_own = M;
  }
  float* out = a.ws + (((size_t)b * a.Hq + kvh * a.g + hj) * a.n_split + split) * kStateFloats;
  const bool writer = view == 0 && hj < a.g;
#pragma unroll
  for (int db = 0; db < 8; ++db) {
    f32x4 o4 = acc_o[db] * W_own;
    if (BIFOCAL) {
#pragma unroll
      for (int i = 0; i < 4; ++i) o4[i] += W_oth * __shfl_xor(acc_o[db][i], 8);
    }
    if (writer) *(f32x4*)(out + 4 + 16 * db + 4 * g4) = o4;
  }
  // the state's third word carries this sequence's split count, so the
  // reduce need not recompute the plan (slot 0 is written by every call)
  if (writer && g4 == 0)
    *(f32x4*)out = f32x4{m_own, W_own * l_own + W_oth * l_oth, __int_as_float(ns), 0.f};
}

// Final merge over the splits of one head (Eq. (7) weights exp2(m - M)):
// O = sum W O~ / sum W l.  Workgroup (head, quarter of the 128 channels):
// 32 groups of 8 threads; group grp takes splits grp, grp + 32, ... (at most
// kRedPerGroup each, loads issued together), thread c of a group owns
// channels 32 quarter + 4c .. +3; partial sums meet in LDS.
constexpr int kRedGroups = 32;
constexpr int kRedPerGroup = 4;  // splits per group: n_split <= 128
__global__ __launch_bounds__(256) void decode_reduce_kernel(DecodeArgs a, uint16_t* o) {
  __shared__ float sMax[kRedGroups];
  __shared__ __attribute__((aligned(16))) float sAcc[kRedGroups][32];
  __shared__ float sDen[kRedGroups];
  const int bh = blockIdx.x;
  const int quarter = blockIdx.y;
  const int tid = threadIdx.x;
  const float* base = a.ws + (size_t)bh * a.n_split * kStateFloats;
  const int c = tid & 7;
  const int grp = tid >> 3;

  // every slot is read at once, slot 0's state carrying the sequence's split
  // count; the slots past it hold stale states and are dropped below
  float m[kRedPerGroup], l[kRedPerGroup];
  f32x4 ov[kRedPerGroup];
#pragma unroll
  for (int i = 0; i < kRedPerGroup; ++i) {
    // no branch: all loads are issued together (slots past n_split read the
    // last slot again and are dropped with the rest)
    const float* stt = base + (size_t)min(grp + kRedGroups * i, a.n_split - 1) * kStateFloats;
    const float2 ml = *(const float2*)stt;
    m[i] = ml.x;
    l[i] = ml.y;
    ov[i] = *(const f32x4*)(stt + 4 + 32 * quarter + 4 * c);
  }
  const int ns = __float_as_int(base[2]);  // splits with keys, from slot 0's state
#pragma unroll
  for (int i = 0; i < kRedPerGroup; ++i) {
    if (grp + kRedGroups * i >= ns) {
      m[i] = -INFINITY;
      l[i] = 0.f;
      ov[i] = f32x4{};
    }
  }
  float M = -INFINITY;
#pragma unroll
  for (int i = 0; i < kRedPerGroup; ++i) M = fmaxf(M, m[i]);
  if (c == 0) sMax[grp] = M;
  __syncthreads();
#pragma unroll
  for (int g2 = 0; g2 < kRedGroups; ++g2) M = fmaxf(M, sMax[g2]);

  f32x4 acc = f32x4{};
  float den = 0.f;
#pragma unroll
  for (int i = 0; i < kRedPerGroup; ++i) {
    const float w = m[i] == -INFINITY ? 0.f : fast_exp2(m[i] - M);
    den += w * l[i];
    acc += w * ov[i];
  }
  *(f32x4*)&sAcc[grp][4 * c] = acc;
  if (c == 0) sDen[grp] = den;
  __syncthreads();
  if (tid < 32) {
    float num = 0.f, dsum = 0.f;
#pragma unroll
    for (int g2 = 0; g2 < kRedGroups; ++g2) {
      num += sAcc[g2][tid];
      dsum += sDen[g2];
    }
    const __bf16 r = (__bf16)(num / dsum);
    o[(size_t)bh * kHeadDim + 32 * quarter + tid] = __builtin_bit_cast(uint16_t, r);
  }
}

// ---------------------------------------------------------------- launcher
// Batches of up to this many sequences get split counts balanced over their
// actual lengths (each workgroup computes the plan from kv_lens, one lane
// per sequence); larger batches split every sequence by max_len.
constexpr int kDecBalancedMaxB = 64;

// About one workgroup per CU (each holds 157 KB of LDS): enough copies in
// flight to stream at full bandwidth while keeping few split states for the
// reduce (at most kRedGroups * kRedPerGroup per head).  Split s takes the
// 16-key steps s, s + ns, ...; *chunk is the most keys one split covers.
void decode_geometry(int B, int Hkv, int max_len, int* chunk, int* n_split) {
  const long long groups = (long long)B * ((Hkv + kDecHeads - 1) / kDecHeads);
  const long long steps = ((long long)max_len + kDecTile - 1) / kDecTile;
  long long want = B <= kDecBalancedMaxB ? kRedGroups * kRedPerGroup : (256 + groups - 1) / groups;
  if (want > kRedGroups * kRedPerGroup) want = kRedGroups * kRedPerGroup;
  if (want > steps) want = steps;
  *n_split = (int)want;
  *chunk = (int)((steps + want - 1) / want * kDecTile);
}

static int cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n < 1)
      n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

size_t decode_workspace_bytes(int B, int Hq, int Hkv, int max_len) {
  int chunk, n_split, n_hgroups;
  decode_geometry(B, Hkv, max_len, &chunk, &n_split);
  return (size_t)B * Hq * n_split * kStateFloats * sizeof(float);
}

size_t decode_map_workspace_bytes(int B, int Hq, int Hkv, int max_len, bool /*freq*/) {
  return decode_workspace_bytes(B, Hq, Hkv, max_len);
}

// block_table == nullptr: dense caches [B][max_len][Hkv][128]; otherwise
// pools [n_pages][1 << page_shift][Hkv][128] and max_len = max_pages << page_shift.
hipError_t launch_decode(bool bifocal, const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                         const int32_t* kv_lens, int max_len, uint16_t* o, const float2* table,
                         int B, int Hq, int Hkv, int w_pre, int w0, float* ws,
                         hipStream_t stream, hipEvent_t ev0, hipEvent_t ev1,
                         const int32_t* block_table, int max_pages, int n_pages, int page_shift,
                         const double* freq_og) {
  // freq_og: nullptr for the Eq. (3) map, else the frequency map's omega_i
  // (64) and ramp gamma_i (64); its rows follow the states in ws
  DecodeArgs a = {};
  a.q = q;
  a.kc = kc;
  a.vc = vc;
  a.kv_lens = kv_lens;
  a.ws = ws;
  a.table = table;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.g = Hq / Hkv;
  a.max_len = max_len;
  a.block_table = block_table;
  a.max_pages = max_pages;
  a.n_pages = n_pages;
  a.page_shift = page_shift;
  decode_geometry(B, Hkv, max_len, &a.chunk, &a.n_split);
  a.n_hgroups = (Hkv + kDecHeads - 1) / kDecHeads;
  a.balanced = B <= kDecBalancedMaxB;
  const int n_cu = cu_count();
  a.n_target = n_cu > B * a.n_hgroups ? n_cu : B * a.n_hgroups;
  a.w_pre = w_pre;
  a.w0 = w0;
  a.q_scale = 1.4426950408889634f / sqrtf((float)kHeadDim);
  const long long nwg = a.balanced ? (long long)a.n_target : (long long)a.n_split * a.n_hgroups * B;
  if (nwg > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  hipError_t e = hipSuccess;
  const bool freq = bifocal && freq_og != nullptr;
  if (freq) {
    for (int i = 0; i < kHalf; ++i) {
      a.fomega[i] = freq_og[i];
      a.fgamma[i] = freq_og[kHalf + i];
    }
  }
  // ev0 / ev1 (optional) are recorded on the stream around the split kernel
  if (ev0 != nullptr && (e = hipEventRecord(ev0, stream)) != hipSuccess) return e;
  if (freq)
    hipLaunchKernelGGL(decode_split_kernel<2>, dim3((unsigned)nwg), dim3(kDecThreads), 0, stream,
                       a);
  else if (bifocal)
    hipLaunchKernelGGL(decode_split_kernel<1>, dim3((unsigned)nwg), dim3(kDecThreads), 0, stream,
                       a);
  else
    hipLaunchKernelGGL(decode_split_kernel<0>, dim3((unsigned)nwg), dim3(kDecThreads), 0, stream,
                       a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (ev1 != nullptr && (e = hipEventRecord(ev1, stream)) != hipSuccess) return e;
  hipLaunchKernelGGL(decode_reduce_kernel, dim3(B * Hq, 4), dim3(256), 0, stream, a, o);
  return hipGetLastError();
}

// ------------------------------------- fixed device scratch (no allocation)
// For callers that cannot allocate device memory (code under graph capture,
// tight serving loops): one file-scope array per device holds the fp32
// cos/sin table of positions [0, kNoAllocMaxLen) and the split states.  The
// array lives as long as the process.  Calls on one device share it, and each
// keeps the last call's contents (the table stays, the states are rewritten
// in full by every call), so calls that overlap on one device race.
constexpr int kNoAllocMaxLen = 1 << 17;
constexpr size_t kNoAllocTableBytes = (size_t)kNoAllocMaxLen * kHalf * sizeof(float2);  // 64 MiB
constexpr size_t kNoAllocStateBytes = (size_t)24 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocTableBytes + kNoAllocStateBytes];

hipError_t launch_build_table(float2* table, uint32_t* table16, int n_pos, const double* omega,
                              hipStream_t stream);

int noalloc_decode_max_len() { return kNoAllocMaxLen; }
size_t noalloc_decode_state_bytes() { return kNoAllocStateBytes; }

namespace {
struct NoAllocDevice {
  unsigned char* ptr = nullptr;  // this device's copy of `scratch`
  double theta = 0.0;            // rope_theta of the table it holds (0: none yet)
};
std::mutex g_noalloc_mu;
NoAllocDevice g_noalloc[64];
}  // namespace

// The current device's table and state regions.  The first call on a device
// looks the array's address up (with that device current); the first call
// for a new theta builds the table from omega and waits for it, so that a
// call on any stream may read it afterwards.
hipError_t noalloc_decode_buffers(double theta, const double* omega, hipStream_t stream,
                                  const float2** table, float** states) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_noalloc_mu);
  NoAllocDevice& d = g_noalloc[dev];
  if (d.ptr == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress((void**)&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    d.ptr = (unsigned char*)p;
  }
  if (d.theta != theta) {
    d.theta = 0.0;
    e = launch_build_table((float2*)d.ptr, nullptr, kNoAllocMaxLen, omega, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return e;
    d.theta = theta;
  }
  *table = (const float2*)d.ptr;
  *states = (float*)(d.ptr + kNoAllocTableBytes);
  return hipSuccess;
}

}  // namespace jl
