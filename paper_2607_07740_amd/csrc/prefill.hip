// prefill.hip -- fused causal bifocal-RoPE attention, prefill, for gfx950.
//
// Jet-Long (arXiv 2607.07740): a key k <= q is scored with the base rotation
// R(q), R(k) when q - k <= w0 and with the remote rotation R(f(q)), R(f(k)),
// f(x) = floor(x / G), otherwise (Sec. 3, Eq. (1); Sec. 3.1, Eqs. (2)-(3)).
// Prefill is the inclusion-exclusion combination of attention passes over the
// two views (Sec. 3.3, Eq. (7)), fused into one kernel.
//
// Launches per call:
//  1. vt_prep_kernel transposes V into the byte image of each 64-key tile that
//     the attention kernel reads in the PV product (a call-scoped buffer; the
//     caller's K and V are only read).
//  2. prefill_kernel, a fast pass and then a checked rerun of the blocks the
//     fast pass listed (see the softmax below), reads raw (pre-RoPE) K tiles from memory straight into
//     registers, 8 keys per wave, with the cos/sin rows of their positions,
//     and rotates them to the view of the visit: k_loc = R(k) x_k on band
//     tiles, k_rem = R(f(k)) x_k on remote tiles (Sec. 3.2, Eqs. (4)-(6): the
//     cache keeps unrotated keys and the rotation is formed on the fly).  The
//     rotated tile lives only in LDS, for the QK product of that visit; no
//     rotated key is ever written to memory.  Each wave rotates its own 8
//     keys, one rotate-half pair of 16-byte chunks per lane.
//
// Work decomposition: a workgroup is 8 wave64s and owns 256 query rows =
// (head hl = r / BQ, position q0 + r % BQ) for the g = Hq/Hkv query heads
// sharing one kv head (GQA packing), BQ = 256 / g.  One workgroup fills a CU
// (two waves per SIMD at 256 VGPRs each; 64 KB of LDS), and each rotated K
// tile and V^T image in LDS serves its 256 rows.  A wave owns 32 rows; a
// lane owns one query column of S^T = K Q^T (v_mfma_f32_32x32x16_bf16, lanes l
// and l + 32 split the column's 16 accumulator rows), and O^T += V^T P^T takes
// P^T straight from the S^T accumulator registers.  Rotated K tiles and V^T
// images of 64-key tiles are double-buffered separately.  The loop is
// software pipelined: while the softmax of tile j runs on the VALU, the QK
// product of tile j+1 is already on the matrix cores, followed by PV of tile
// j; meanwhile each wave copies its share of V(j+1) into LDS and rotates its
// 8 keys of K(j+2).  The O^T accumulator (4 x 16 fp32 per lane) stays in
// VGPRs, and each segment's loop is unrolled twice so the two score buffers
// alternate without copies.
//
// Softmax runs in the log2 domain against a per-row reference m (initially 0)
// that the QK product subtracts itself: its first k-step accumulates onto -m.
// The common path is exp2, convert and a dot product for the row sum.  A
// first, fast pass never moves the reference: it only notes, per tile, whether
// a row's probability sum passed 2^64 and, at the end, whether a row's total
// fell below 2^-64; a block that trips either writes nothing and is listed.
// A second launch reruns the listed blocks with the checked kernel, which
// tests each tile's probability sum after its softmax and, in a rare branch,
// moves the reference to the tile's largest score (when that lies more than 64
// above it, or more than 64 below it before anything was accumulated),
// re-bases the tile and rescales the state.  So every probability stays below
// 2^64.
#include <climits>
#include <type_traits>

#include "jl_device.h"

namespace jl {

constexpr int kPfWaves = 8;             // waves per workgroup: two per SIMD
constexpr int kPfThreads = 64 * kPfWaves;
constexpr int kPfRows = 32 * kPfWaves;  // query rows per workgroup: 32 per wave
constexpr int kPfBK = 64;               // keys per tile
constexpr int kTileBytes = kPfBK * kHeadDim * 2;  // one K tile or one V^T image: 16 KB
// LDS: rotated K tiles (two buffers) and V^T images (two)
constexpr int kRotOff = 0, kVtOff = 2 * kTileBytes;
constexpr int kSmemBytes = 4 * kTileBytes;  // 64 KB
constexpr int kPfCopyBytes = kTileBytes / kPfWaves;  // each wave's share of a tile copy: 8 keys
constexpr int kKeysPerWave = kPfBK / kPfWaves;
constexpr int kRetryCounters = 3;  // rerun counters at the head of the rerun area

// LDS layouts.
//   rotated K tile: key r (0..63) at r * 256; its 16-byte
//              chunk c (d = 8c .. 8c+7) sits in slot c ^ kswz(r), with
//              kswz(r) = (r & 15) >> 1 | (r & 1) << 3 a permutation of 0..15.
//              16 lanes reading 16 consecutive keys at one chunk (the QK
//              operand reads) hit 16 distinct bank groups, and so do 16 lanes
//              covering chunks 0..7 (or 8..15) of an even and the following
//              odd key (the rotation's writes).
//   (The raw keys and their cos/sin rows go from memory to registers and
//   never pass through LDS.)
//   V^T image: d (0..127) at d * 128; slot s of a row holds the 8 keys of
//              group g = s ^ ((d >> 1) & 7), g = 2 ks + h, in the order
//              t -> key 16 ks + 8 (t / 4) + 4 h + t % 4 (the k order of the
//              P^T operand, i.e. of the S^T accumulator rows).  16 lanes
//              reading 16 consecutive d at one group hit 16 distinct groups.
__device__ inline int kswz(int r) { return ((r & 15) >> 1) | ((r & 1) << 3); }
__device__ inline int kimg_off(int r, int c) { return r * 256 + 16 * (c ^ kswz(r)); }
__device__ inline int vtimg_off(int d, int g) { return d * 128 + 16 * (g ^ ((d >> 1) & 7)); }

struct PrepArgs {
  const uint16_t* v;
  uint16_t* vt;  // [B][Hkv][n_tiles] V^T images
  int B, Hkv, L, n_tiles;  // L: keys [0, L) are valid
  int kv_stride;           // rows per sequence in v (>= L)
  // packed variable-length batches: per tile (seq0, L, tile, tile0) with
  // seq0 the sequence's first row of v and tile0 its first tile; the images
  // of kv head h sit at (h * n_tiles + tile0 + tile).  nullptr for dense
  // batches.
  const int4* twork;
  int* retry_count;  // zeroed here for the attention kernel that follows
  // paged caches (nullptr otherwise): v is a pool [n_pages][page][Hkv][128]
  // and key k of sequence b sits in page block_table[b][k >> page_shift]
  const int32_t* block_table;
  int max_pages, page_shift, n_pages;
};

// Pool row of key k0 (the first key of a tile; pages hold whole tiles) in
// page `page`, clamped into the pool.
__device__ inline size_t paged_row(int page, int n_pages, int page_shift, int k0) {
  page = page < 0 ? 0 : (page >= n_pages ? n_pages - 1 : page);
  return ((size_t)page << page_shift) + (size_t)(k0 & ((1 << page_shift) - 1));
}

// One workgroup per (tile, b * Hkv + kvh), or per (tile work item, kvh) for a
// packed batch.  Keys past the sequence's length are written as zeros.
__global__ __launch_bounds__(256) void vt_prep_kernel(PrepArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sv[kPfBK * kHeadDim];
  // the rerun counters: one per attention pass that follows (the literal
  // mode's three window passes use three)
  if (a.retry_count != nullptr && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x < kRetryCounters)
    a.retry_count[threadIdx.x] = 0;
  int tile, L;
  size_t seq_row, img;
  const int kvh_v = blockIdx.y;
  if (a.twork != nullptr) {
    const int4 w = a.twork[blockIdx.x];
    if (w.y <= 0) return;  // no tile here (uniform, before any barrier)
    tile = w.z;
    L = w.y;
    seq_row = (size_t)w.x;
    img = ((size_t)kvh_v * a.n_tiles + w.w + tile) * (kTileBytes / 2);
  } else {
    tile = blockIdx.x;
    L = a.L;
    const int b = blockIdx.y / a.Hkv;
    seq_row = (size_t)b * a.kv_stride;
    img = ((size_t)blockIdx.y * a.n_tiles + tile) * (kTileBytes / 2);
  }
  const int kvh = a.twork != nullptr ? kvh_v : (int)(blockIdx.y % a.Hkv);
  const int t = threadIdx.x;
  const int k0 = tile * kPfBK;
  const size_t row = (size_t)a.Hkv * kHeadDim;
  // the tile's first key row: paged pools hold whole tiles in a page
  size_t trow = seq_row + k0;
  if (a.block_table != nullptr) {
    const int b = blockIdx.y / a.Hkv;
    trow = paged_row(a.block_table[(size_t)b * a.max_pages + (k0 >> a.page_shift)], a.n_pages,
                     a.page_shift, k0);
  }
  const uint16_t* vtile = a.v + (trow * a.Hkv + kvh) * kHeadDim;

  // V tile -> LDS, zeros past L
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int idx = t + 256 * i;  // 64 keys x 16 chunks
    const int r = idx >> 4, c = idx & 15;
    u32x4 w = u32x4{0, 0, 0, 0};
    if (k0 + r < L) w = load16(vtile + (size_t)r * row + 8 * c);
    *(u32x4*)(sv + r * kHeadDim + 8 * c) = w;
  }
  __syncthreads();

  // V^T: 128 d x 8 key groups of 16 bytes, 4 per thread
  unsigned char* vti = (unsigned char*)(a.vt + img);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int p = t + 256 * i;
    const int d = p >> 3, g = p & 7;
    const int ks = g >> 1, h = g & 1;
    uint16_t e[8];
#pragma unroll
    for (int tt = 0; tt < 8; ++tt) e[tt] = sv[(16 * ks + 8 * (tt >> 2) + 4 * h + (tt & 3)) * kHeadDim + d];
    u32x4 w;
#pragma unroll
    for (int q = 0; q < 4; ++q) w[q] = (unsigned)e[2 * q] | ((unsigned)e[2 * q + 1] << 16);
    *(u32x4*)(vti + vtimg_off(d, g)) = w;
  }
}

struct PrefillArgs {
  const uint16_t* q;
  uint16_t* o;
  float* lse;
  const float2* table;   // [positions][64] (cos, sin) of p * omega_i
  const float2* rtable;  // remote view: table read at f(p), or the frequency map's table at p
  const uint32_t* table16;   // the same tables as bf16 pairs (cos low, sin high): key rotation
  const uint32_t* rtable16;
  int freq_map;          // 0: Eq. (3) aliasing, 1: Sec. 4.5 frequency interpolation
  int rtab_packed;       // packed batch with the frequency map: the remote tables hold
                         // each sequence's own rows, from the sequence's first row on
  const uint16_t* k;     // raw (pre-RoPE) keys, [B][kv_stride][Hkv][128] or packed [T][Hkv][128]
  const uint16_t* vt;    // V^T tile images from vt_prep_kernel
  int kv_stride;         // rows per sequence in k (dense batches)
  int B, Hq, Hkv, L, n_tiles;  // L: keys [0, L), the call's sequence length (G follows it)
  int q_start, Lq;              // query rows: positions q_start .. q_start + Lq - 1 (= L - Lq ..)
  int g, BQ, n_qblocks;
  int w0;         // local window; INT_MAX for the vanilla kernel and window B
  FastDiv gdiv;   // division by G (Eq. (3))
  float q_scale;  // log2(e) / sqrt(head_dim): scores come out in log2 units
  float slack;    // log2 units a tile maximum may lie above (or, before anything
                  // was accumulated, below) the reference before it moves (64)
  float* o32;     // window passes: normalised fp32 O_X [B][L][Hq][128]
  // packed variable-length batch (nullptr otherwise): one (seq0, L, q block,
  // tile0) per Hkv consecutive workgroups; q and o are [T][Hq][128] with
  // T = Lq, lse is [Hq][T], the sequence's tile images start at tile0 and
  // each sequence takes its own G = group_size(L, w_pre)
  const int4* qwork;
  int w_pre;
  // blocks whose fast pass needs the reference check (see prefill_kernel):
  // a counter and the workgroup indices; nullptr where unused
  int* retry_count;
  int* retry_list;
  // paged caches (nullptr otherwise): k is a pool [n_pages][page][Hkv][128],
  // pages of at least 64 keys, so a tile lies in one page
  const int32_t* block_table;
  int max_pages, page_shift, n_pages;
};

// Most pages of one sequence a paged prefill block looks up (LDS table)
constexpr int kMaxSeqPages = 4096;

// One workgroup's query block: workgroup -> (b, kv head, q block), longest
// q blocks first.  When the (b, kv head) groups are a multiple of the 8 XCDs,
// consecutive work items land on one XCD so a group's K/V tiles stay in that
// XCD's L2.  A packed batch reads its work item from the plan instead.
struct Work {
  int b, kvh, qblk, q_start, q_end, w0, Lk;  // Lk: keys [0, Lk) of the sequence are valid
  size_t row_base, lse_base, img_base;    // rows of q/o, lse entries, V^T image elements
  size_t kv_row0;                         // the sequence's first row of k
  size_t rtab_row;                        // the sequence's row 0 in the remote tables
  FastDiv gdiv;
};

// false: no query block here (an unused entry of a packed batch's plan)
__device__ inline bool work_of(const PrefillArgs& a, int bid, bool fused, Work& W) {
  const int n_groups = a.B * a.Hkv;
  if (a.qwork != nullptr) {
    // packed batch: the work item's sequence, its G, its tiles; the kv head
    // follows the XCD (bid & 7) when Hkv divides 8
    const int item = bid / a.Hkv;
    W.b = 0;
    W.kvh = bid - item * a.Hkv;
    const int4 w = a.qwork[item];
    if (w.y <= 0) return false;
    const int G = fused ? group_size(w.y, a.w_pre) : 1;
    W.gdiv = make_fastdiv((uint32_t)G);
    W.w0 = G > 1 ? a.w0 : INT_MAX;  // G = 1: the unmodified model, as the dense call
    W.qblk = w.z;
    W.q_start = 0;
    W.q_end = w.y;
    W.row_base = (size_t)w.x;
    W.lse_base = (size_t)w.x;
    W.img_base = ((size_t)W.kvh * a.n_tiles + w.w) * (kTileBytes / 2);
    W.kv_row0 = (size_t)w.x;
    W.rtab_row = a.rtab_packed ? (size_t)w.x : 0;
    W.Lk = w.y;
  } else {
    int group;
    if ((n_groups & 7) == 0) {
      const int work = (bid & 7) * (gridDim.x >> 3) + (bid >> 3);
      group = work / a.n_qblocks;
      W.qblk = a.n_qblocks - 1 - (work - group * a.n_qblocks);
    } else {
      W.qblk = a.n_qblocks - 1 - bid / n_groups;
      group = bid - (bid / n_groups) * n_groups;
    }
    const int b = group / a.Hkv;
    W.b = b;
    W.kvh = group - b * a.Hkv;
    W.gdiv = a.gdiv;
    W.w0 = a.w0;
    W.q_start = a.q_start;
    W.q_end = a.q_start + a.Lq;  // one past the last query position
    W.row_base = (size_t)b * a.Lq;
    W.lse_base = (size_t)b * a.Hq * a.Lq;
    W.img_base = (size_t)group * a.n_tiles * (kTileBytes / 2);
    W.kv_row0 = (size_t)b * a.kv_stride;
    W.rtab_row = 0;
    W.Lk = a.L;
  }
  return true;
}

// What one launch of the attention kernel computes.
//   kModeFused    the bifocal result in one pass: remote-view tiles holding
//                 pairs with q - k > w0, then base-view tiles of the band
//   kModeVanilla  causal attention in the base view (the unmodified model)
//   kModeWinA/B/C the three attention calls of Eq. (7), each a single view
//                 over one key set: A = band in the base view, B = all causal
//                 keys in the remote view, C = band in the remote view.
//                 They write normalised fp32 O_X and the natural-log LSE_X.
enum PrefillMode : int { kModeFused = 0, kModeVanilla = 1, kModeWinA = 2, kModeWinB = 3, kModeWinC = 4 };

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
__device__ inline bf16x2 bf16_one2() { return bf16x2{(__bf16)1.0f, (__bf16)1.0f}; }

// Load one query row's B operand: 8 k-steps of 8 bf16 (d = 16 s + 8 half + j),
// rotated to position pos and scaled.  Pairs (s, s + 4) are rotate-half partners.
__device__ inline void load_q_operand(const uint16_t* qrow, int half, const float2* table,
                                      int pos, float scale, bf16x8* out) {
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int d = 16 * s + 8 * half;
    float lo[8], hi[8], ylo[8], yhi[8];
    unpack8(load16(qrow + d), lo);
    unpack8(load16(qrow + d + kHalf), hi);
    const float4* c4 = (const float4*)(table + (size_t)pos * kHalf + d);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const float4 w = c4[t];  // (cos_i, sin_i, cos_{i+1}, sin_{i+1})
      const int j = 2 * t;
      ylo[j] = (lo[j] * w.x - hi[j] * w.y) * scale;
      yhi[j] = (hi[j] * w.x + lo[j] * w.y) * scale;
      ylo[j + 1] = (lo[j + 1] * w.z - hi[j + 1] * w.w) * scale;
      yhi[j + 1] = (hi[j + 1] * w.z + lo[j + 1] * w.w) * scale;
    }
    out[s] = pack8(ylo);
    out[s + 4] = pack8(yhi);
  }
}


// SAFE = false (fused and vanilla modes): the fast pass.  It never waits on
// the softmax reference check; instead it records, without a branch, whether
// any tile's probability sum exceeded 2^slack, and at the end whether a row's
// total fell below 2^-slack.  A block with either writes nothing and lists
// itself; the SAFE launch that follows reruns only the listed blocks with the
// per-tile check, which moves the reference as needed.  Every mode runs so.
template <int MODE, bool SAFE, bool PAGED = false>
__global__ __launch_bounds__(kPfThreads, 2) void prefill_kernel(PrefillArgs a) {
  constexpr bool CHECK_LATE = !SAFE;
  // The visit list has at most two segments: the fused kernel's remote tiles
  // (segment 1), then tiles [kt_l, n_kt) in one view, keeping 0 <= q - k <= w0
  // (segment 2; w0 = INT_MAX makes it the causal set).
  constexpr bool FUSED = MODE == kModeFused;
  constexpr bool REMOTE2 = MODE == kModeWinB || MODE == kModeWinC;  // segment 2's view
  constexpr bool OUT_F32 = MODE == kModeWinA || MODE == kModeWinB || MODE == kModeWinC;
  constexpr bool FROM_ZERO = MODE == kModeVanilla || MODE == kModeWinB;  // kt_l = 0
  // LDS: raw K tiles, rotated K tiles and V^T images, two buffers each
  __shared__ __attribute__((aligned(1024))) unsigned char smem[kSmemBytes];
  __shared__ int s_bad;
  __shared__ int s_pages[PAGED ? kMaxSeqPages : 1];  // paged caches: the sequence's pages

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int hl32 = lane >> 5;  // which 8-wide half of a 16-wide k slice this lane feeds

  int bid = blockIdx.x;
  if (SAFE && a.retry_list != nullptr) {  // rerun of the listed blocks only
    if (bid >= *a.retry_count) return;    // uniform, before any barrier
    bid = a.retry_list[bid];
  }
  Work W;
  if (!work_of(a, bid, FUSED, W)) return;  // uniform, before any barrier
  const int kvh = W.kvh, qblk = W.qblk, q_start = W.q_start, q_end = W.q_end, w0 = W.w0, Lk = W.Lk;
  const size_t row_base = W.row_base, lse_base = W.lse_base, img_base = W.img_base;
  const size_t kv_row0 = W.kv_row0;
  const float2* rtable = a.rtable + W.rtab_row * kHalf;
  const uint32_t* rtable16 = a.rtable16 + W.rtab_row * kHalf;
  const FastDiv gdiv = W.gdiv;
  const int q0 = q_start + qblk * a.BQ;
  const int q1 = min(q0 + a.BQ, q_end) - 1;

  // ---- this lane's query row: column (lane & 31) of the wave's 32
  const int row = 32 * wave + (lane & 31);
  const int hl = row / a.BQ;
  const int qpos = q0 + (row - hl * a.BQ);
  const bool row_valid = qpos < q_end;
  const int qp = row_valid ? qpos : q_end - 1;
  const int hd = kvh * a.g + hl;
  const int qr = qp - q_start;  // row of this query in its sequence's q, o and lse
  const uint16_t* qrow = a.q + ((row_base + qr) * a.Hq + hd) * kHeadDim;

  // ---- visit list: segment 1 = tiles [0, n_r), segment 2 = tiles [kt_l, n_kt)
  const VisitRanges vr = visit_ranges(q0, q1, w0, kPfBK);
  const int n_kt = vr.n_kt;
  const int n_r = FUSED ? vr.n_r : 0;
  const int kt_l = FROM_ZERO ? 0 : vr.kt_l;
  const int n_steps = n_r + (n_kt - kt_l);

  // ---- staging.  For list entry j each wave copies its eighth (2 KB) of the
  // V^T image into buffer jb & 1, and rotates 8 keys of the raw K tile, read
  // from memory, into the rotated buffer of that parity.
  const uint32_t smem_base = lds_addr(smem);
  const uint32_t lane_off = 16 * lane;
  auto tile_of = [&](int j) __attribute__((always_inline)) { return j < n_r ? j : kt_l + (j - n_r); };
  // j's view: remote (R(f(k)), Eq. (3), or the frequency map's table at k) or base (R(k))
  auto is_remote = [&](int j) __attribute__((always_inline)) { return REMOTE2 || (FUSED && j < n_r); };
  // Scalar description of list entry j, formed a visit before its
  // rotation.  The cos/sin rows of a
  // tile are contiguous: p(k0) .. p(min(k0 + 63, Lk - 1)) with p = f for the
  // aliasing remote view (at most 32 rows, as G >= 2 there) and the identity
  // otherwise (64 rows); key k0 + r reads row f(k0 + r) - f(k0) =
  // floor((kmod + r) / G), kmod = k0 - G f(k0), or row r.  f is formed on
  // every entry and selected, so no branch splits the loop body (the
  // remote-view kernels run with G >= 2).
  struct Ent {
    int k0, klim;  // first key; Lk - 1 - k0 (rows past it repeat the last key)
    int row0, tlim;  // first cos/sin row; index of the last valid row
    int kmod;
    int alias, remote;
  };
  const uint32_t G_d = gdiv.d;
  auto ent_of = [&](int j) __attribute__((always_inline)) {
    Ent e;
    e.k0 = tile_of(j) * kPfBK;
    e.klim = Lk - 1 - e.k0;
    e.remote = is_remote(j);
    e.alias = e.remote & (a.freq_map == 0);
    uint32_t f0 = fastdiv_ge2((uint32_t)e.k0, gdiv);
    const int nlast = min(kPfBK - 1, e.klim);
    uint32_t km = (uint32_t)e.k0 - G_d * f0;
    uint32_t fl = fastdiv_ge2(km + (uint32_t)nlast, gdiv);
    asm volatile("" : "+s"(f0), "+s"(km), "+s"(fl));
    e.row0 = e.alias ? (int)f0 : e.k0;
    e.kmod = e.alias ? (int)km : 0;
    e.tlim = e.alias ? (int)fl : nlast;
    return e;
  };
  const size_t kseq_off = (kv_row0 * a.Hkv + kvh) * kHeadDim;  // the sequence's key 0 in k
  auto issue_v = [&](int j, int jb) __attribute__((always_inline)) {
    const size_t off = img_base + (size_t)tile_of(j) * (kTileBytes / 2) + wave * (kPfCopyBytes / 2);
    const unsigned char* gv = (const unsigned char*)(a.vt + off);
    const uint32_t l = smem_base + kVtOff + (jb & 1) * kTileBytes + wave * kPfCopyBytes;
    dma16_s<0>(gv, lane_off, l);
    dma16_s<1024>(gv, lane_off, l);
  };
  // Rotation of an entry's raw K tile to its view (Sec. 3.2): lane -> key
  // rt_row of the tile, rotate-half pairs of chunks (rt_c, rt_c + 8), i.e.
  // frequencies i = 8 rt_c .. 8 rt_c + 7, with the (cos, sin) of the key's
  // position.  The raw chunks and the cos/sin row go from memory straight
  // into registers (rows past the sequence repeat its last key).  Each output
  // is one v_dot2_f32_bf16 of the pair (x_i, x_{i+64}) with (cos, -sin) or of
  // (x_{i+64}, x_i) with (cos, sin): exact products, an fp32 sum, then one
  // rounding to bf16.  The result exists only in LDS.
  const int rt_row = kKeysPerWave * wave + (lane >> 3);
  const int rt_c = lane & 7;
  const int rt_lo = kimg_off(rt_row, rt_c), rt_hi = kimg_off(rt_row, rt_c + 8);
  struct RotIn {
    u32x4 xl, xh;  // raw chunks rt_c and rt_c + 8 of key rt_row
    u32x4 ca, cb;  // bf16 (cos, sin) of frequencies 8 rt_c .. +3 and +4 .. +7
  };
  auto rot_load = [&](const Ent& e) __attribute__((always_inline)) {
    int fr = (int)fastdiv_ge2((uint32_t)(e.kmod + rt_row), gdiv);
    asm volatile("" : "+v"(fr));  // formed unconditionally: a select, not a branch
    const int row = min(e.alias ? fr : rt_row, e.tlim);
    const int key = min(rt_row, e.klim);
    const uint16_t* kr;
    if constexpr (PAGED) {  // the tile's page (clamped already; a page holds whole tiles)
      const int page = __builtin_amdgcn_readfirstlane(s_pages[e.k0 >> a.page_shift]);
      const size_t prow = ((size_t)page << a.page_shift) + (e.k0 & ((1 << a.page_shift) - 1));
      kr = a.k + ((prow + key) * a.Hkv + kvh) * kHeadDim;
    } else {
      kr = a.k + kseq_off + (size_t)(e.k0 + key) * ((size_t)a.Hkv * kHeadDim);
    }
    const uint32_t* tr =
        (e.remote ? rtable16 : a.table16) + (size_t)(e.row0 + row) * kHalf + 8 * rt_c;
    RotIn r;
    r.xl = load16(kr + 8 * rt_c);
    r.xh = load16(kr + 64 + 8 * rt_c);
    r.ca = load16(tr);
    r.cb = load16(tr + 4);
    return r;
  };
  // word w (0..3) of the rotated chunks: frequencies 8 rt_c + 2w and + 1
  auto rot_word = [&](const RotIn& r, int w, u32x4& lo, u32x4& hi) __attribute__((always_inline)) {
    const uint32_t cs_a = w < 2 ? r.ca[2 * w] : r.cb[2 * w - 4];
    const uint32_t cs_b = w < 2 ? r.ca[2 * w + 1] : r.cb[2 * w - 3];
    uint32_t l, h;
    rot_word_dot2(r.xl[w], r.xh[w], cs_a, cs_b, l, h);
    lo[w] = l;
    hi[w] = h;
  };
  auto rot_store = [&](int jb, const u32x4& lo, const u32x4& hi) __attribute__((always_inline)) {
    unsigned char* dst = smem + kRotOff + (jb & 1) * kTileBytes;
    *(u32x4*)(dst + rt_lo) = lo;
    *(u32x4*)(dst + rt_hi) = hi;
  };
  auto rotate = [&](const RotIn& r, int jb) __attribute__((always_inline)) {
    u32x4 lo, hi;
#pragma unroll
    for (int w = 0; w < 4; ++w) rot_word(r, w, lo, hi);
    rot_store(jb, lo, hi);
  };
  auto kbuf = [&](int j) __attribute__((always_inline)) {
    return (const unsigned char*)smem + kRotOff + (j & 1) * kTileBytes;
  };
  auto vbuf = [&](int j) __attribute__((always_inline)) {
    return (const unsigned char*)smem + kVtOff + (j & 1) * kTileBytes;
  };

  // ---- state.  Scores are log2-domain (q_scale folded into Q) and come out
  // of the MFMA already relative to a per-row reference m_ref: the first
  // k-step of every QK product accumulates onto neg_m = -m_ref in each entry
  // (all 16 accumulator entries of a lane belong to its query column).  The
  // reference moves only on the rare path below.
  bf16x8 qop[8];
  f32x16 acc_o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc_o[i] = f32x16{};
  float m_ref = 0.f;
  f32x16 neg_m = f32x16{};
  float l_run = 0.f;
  f32x16 sc_a[2], sc_b[2];

  const int kr_lane = lane & 31;
  // S^T = K Q^T for one tile: 2 blocks of 32 keys x 8 k-steps.  The two
  // blocks' accumulation chains alternate so that consecutive MFMAs are
  // independent; K operands are read 4 MFMAs ahead.
  auto qk = [&](const unsigned char* kb, f32x16* sc) __attribute__((always_inline)) {
    auto kop = [&](int m) __attribute__((always_inline)) {
      const int r = 32 * (m & 1) + kr_lane;
      return *(const bf16x8*)(kb + kimg_off(r, 2 * (m >> 1) + hl32));
    };
    bf16x8 ring[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) ring[m] = kop(m);
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      const int blk = m & 1, s = m >> 1;
      sc[blk] = mfma32(ring[m & 3], qop[s], s == 0 ? neg_m : sc[blk]);
      if (m + 4 < 16) ring[m & 3] = kop(m + 4);
    }
  };
  // O^T += V^T P^T: 4 k-steps of 16 keys x 4 d-blocks of 32, V^T operands
  // read 4 MFMAs ahead
  auto pv = [&](const unsigned char* vb, const bf16x8* pb) __attribute__((always_inline)) {
    auto vop = [&](int m) __attribute__((always_inline)) {
      const int d = 32 * (m & 3) + kr_lane;
      return *(const bf16x8*)(vb + vtimg_off(d, 2 * (m >> 2) + hl32));
    };
    bf16x8 ring[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) ring[m] = vop(m);
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      acc_o[m & 3] = mfma32(ring[m & 3], pb[m >> 2], acc_o[m & 3]);
      if (m + 4 < 16) ring[m & 3] = vop(m + 4);
    }
  };

  // Element masks where tile j is not wholly inside its visit's key set.  The
  // fast pass sets each segment's unmasked run [lo, hi] when the segment
  // starts: segment 1 tiles before m1 hold remote pairs only, segment 2
  // tiles t with 64 t >= q1 - w0 and 64 t + 63 <= q0 hold band pairs only.
  // The checked pass tests each tile (fewer live registers).
  auto need_mask = [&](int j) __attribute__((always_inline)) {
    const int k0 = tile_of(j) * kPfBK;
    return j < n_r ? !(q0 - (k0 + kPfBK - 1) > w0) : !(q1 - k0 <= w0 && k0 + kPfBK - 1 <= q0);
  };
  auto seg1_bounds = [&](int& lo, int& hi) __attribute__((always_inline)) {
    const long long x = (long long)q0 - (kPfBK - 1) - w0;  // tile j fully remote: 64 j < x
    lo = 0;
    hi = (x > 0 ? (int)((x + kPfBK - 1) / kPfBK) : 0) - 1;
  };
  auto seg2_bounds = [&](int& lo, int& hi) __attribute__((always_inline)) {
    const long long y = (long long)q1 - w0;
    const int t_lo = y > 0 ? (int)((y + kPfBK - 1) / kPfBK) : 0;
    const int t_hi = q0 >= kPfBK - 1 ? (q0 - (kPfBK - 1)) / kPfBK : -1;
    lo = n_r + t_lo - kt_l;
    hi = n_r + t_hi - kt_l;
  };
  auto mask = [&](int j, f32x16* sc) __attribute__((always_inline)) {
    // keep iff lo <= q - k <= hi: segment 1 keeps q - k > w0, segment 2
    // keeps 0 <= q - k <= w0; one unsigned compare per element
    const bool seg1 = j < n_r;
    const int k0 = tile_of(j) * kPfBK;
    const int lo = seg1 ? w0 + 1 : 0;
    const uint32_t span = seg1 ? (uint32_t)(INT_MAX - lo) : (uint32_t)w0;
    const int base = qp - k0 - lo - 4 * hl32;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const uint32_t off = (uint32_t)(base - (32 * blk + 8 * (i >> 2) + (i & 3)));
        sc[blk][i] = off <= span ? sc[blk][i] : -INFINITY;
      }
    }
  };

  // P^T operands and their row sum: the sum of the rounded probabilities the
  // PV product uses, by dot products of their bf16 pairs in two chains (even
  // and odd pairs), in the order the fast pass forms it, so a block that needs
  // no reference move gets the same l from either pass.  The scores are
  // already relative to the reference.
  auto softmax = [&](const f32x16* sc, bf16x8* pb) __attribute__((always_inline)) {
    float ps0 = 0.f, ps1 = 0.f;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float p[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) p[t] = fast_exp2(sc[q >> 1][8 * (q & 1) + t]);
      pb[q] = pack8(p);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const bf16x2 pair = {pb[q][2 * u], pb[q][2 * u + 1]};
        if (u & 1)
          ps1 = __builtin_amdgcn_fdot2_f32_bf16(pair, bf16_one2(), ps1, false);
        else
          ps0 = __builtin_amdgcn_fdot2_f32_bf16(pair, bf16_one2(), ps0, false);
      }
    }
    return ps0 + ps1;
  };
  // Reference check, after the tile's softmax: the reference moves when a
  // tile probability in a column could exceed 2^slack (their sum does: exp2
  // could overflow), or, before anything was accumulated, when the tile's
  // probabilities sum below 2^-slack (everything could underflow).  The
  // common path is one compare of the sum the softmax already formed and one
  // ballot; the rare path settles each column's maximum (both lane halves),
  // re-bases the tile's scores and the next tile's (computed against the old
  // reference), rescales the running state and redoes the tile's softmax.
  const float p_hi = exp2f(a.slack), p_lo = exp2f(-a.slack);
  unsigned long long late_bad = 0;
  auto ref_fix = [&](f32x16* sc, f32x16* nx, bf16x8* pb, float& ps) __attribute__((always_inline)) {
    const bool bad = ps > p_hi || (l_run == 0.f && ps < p_lo);
    if (__ballot(bad) == 0) return;
    float mt = -INFINITY;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int i = 0; i < 16; ++i) mt = fmaxf(mt, sc[blk][i]);
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float lc = l_run + __shfl_xor(l_run, 32);
    const bool upd = mt != -INFINITY && (mt > a.slack || (lc == 0.f && mt < -a.slack));
    if (__ballot(upd) == 0) return;
    const float shift = upd ? mt : 0.f;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      sc[blk] -= shift;
      nx[blk] -= shift;
    }
    // a downward move only happens before anything was accumulated (lc == 0)
    const float alpha = lc == 0.f ? 1.f : fast_exp2(-shift);
    if (__ballot(upd && lc != 0.f) != 0) {
#pragma unroll
      for (int db = 0; db < 4; ++db) acc_o[db] *= alpha;
    }
    l_run *= alpha;
    m_ref += shift;
#pragma unroll
    for (int i = 0; i < 16; ++i) neg_m[i] = -m_ref;
    ps = softmax(sc, pb);
  };

  // One pipelined visit: on entry `cur` holds the scores of tile j, the
  // rotated K of list entry j+1 is in LDS, and this wave's copies of raw
  // K(j+2) (with its cos/sin rows) and V(j) are in flight.  The QK product of
  // entry j+1 is issued next to the softmax of tile j, then PV of tile j; raw
  // K(j+3) and V(j+1) are copied meanwhile and raw K(j+2) is rotated.  For the last tile of a
  // segment the QK product reads whatever the next K buffer holds and is
  // discarded.
  // pend describes entry j+2 (formed when its copies were issued); on return
  // it describes entry j+3.
  auto visit = [&](int j, f32x16* cur, f32x16* nxt, int lo, int hi, Ent& pend) __attribute__((always_inline)) {
    if (SAFE ? need_mask(j) : (j < lo || j > hi)) mask(j, cur);
    wait_vmem();      // this wave's copy of V(j)
    __syncthreads();  // everyone's; QK(j), PV(j-1) and the rotation of j+1 are done everywhere
    bf16x8 pb[4];
    // V(j+1) into the buffer PV(j-1) released
    issue_v(min(j + 1, n_steps - 1), j + 1);
    if constexpr (!SAFE) {
      // raw K(j+2) and its cos/sin row into registers: they land while
      // QK(j+1) and the softmax of j run
      const RotIn rin = rot_load(pend);
      // The visit is written as two streams cut by scheduling barriers: each
      // MFMA of the QK product of j+1 with its operand read and one
      // sixteenth of the softmax of j (two probabilities, and the bf16 pair
      // of the previous sixteenth); each MFMA of the PV product of j with its
      // operand read, one bf16 pair's dot product for the row sum and, on
      // four of them, a quarter of the rotation of j+2.  The barriers keep
      // the operand reads and the rotation quarters in place.  The pure
      // arithmetic is placed before them, by instruction selection: the
      // exp2 and conversions come together after the QK product's MFMAs and
      // the row-sum dot products after the PV product.  Forcing the written
      // interleave with empty asm ties on each result measured 3% slower on
      // gfx950, and so did leaving the rotation to the compiler as well.
      const unsigned char* kb = kbuf(j + 1);
      auto kop = [&](int m) __attribute__((always_inline)) {
        const int r = 32 * (m & 1) + kr_lane;
        return *(const bf16x8*)(kb + kimg_off(r, 2 * (m >> 1) + hl32));
      };
      bf16x8 ring[4];
#pragma unroll
      for (int m = 0; m < 4; ++m) ring[m] = kop(m);
      bf16x2 pw[16];
      float e0 = 0.f, e1 = 0.f;
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        const int blk = m & 1, st = m >> 1;
        nxt[blk] = mfma32(ring[m & 3], qop[st], st == 0 ? neg_m : nxt[blk]);
        if (m + 4 < 16) ring[m & 3] = kop(m + 4);
        const int q = m >> 2, t = 2 * (m & 3);
        const float p0 = fast_exp2(cur[q >> 1][8 * (q & 1) + t]);
        const float p1 = fast_exp2(cur[q >> 1][8 * (q & 1) + t + 1]);
        if (m > 0) pw[m - 1] = __builtin_convertvector((f32x2){e0, e1}, bf16x2);
        e0 = p0;
        e1 = p1;
        __builtin_amdgcn_sched_barrier(0);
      }
      pw[15] = __builtin_convertvector((f32x2){e0, e1}, bf16x2);
#pragma unroll
      for (int q = 0; q < 4; ++q)
        pb[q] = (bf16x8){pw[4 * q][0], pw[4 * q][1], pw[4 * q + 1][0], pw[4 * q + 1][1],
                         pw[4 * q + 2][0], pw[4 * q + 2][1], pw[4 * q + 3][0], pw[4 * q + 3][1]};
      // past the list's end the last entry is rotated (and V copied) again
      const Ent e3 = ent_of(min(j + 3, n_steps - 1));
      const unsigned char* vb = vbuf(j);
      auto vop = [&](int m) __attribute__((always_inline)) {
        const int d = 32 * (m & 3) + kr_lane;
        return *(const bf16x8*)(vb + vtimg_off(d, 2 * (m >> 2) + hl32));
      };
#pragma unroll
      for (int m = 0; m < 4; ++m) ring[m] = vop(m);
      // the rotated words in units 1, 4, 7, 10; stored early, so the writes
      // are done well before the next barrier
      u32x4 rlo, rhi;
      float ps0 = 0.f, ps1 = 0.f;
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        acc_o[m & 3] = mfma32(ring[m & 3], pb[m >> 2], acc_o[m & 3]);
        if (m + 4 < 16) ring[m & 3] = vop(m + 4);
        if (m & 1)
          ps1 = __builtin_amdgcn_fdot2_f32_bf16(pw[m], bf16_one2(), ps1, false);
        else
          ps0 = __builtin_amdgcn_fdot2_f32_bf16(pw[m], bf16_one2(), ps0, false);
        if (m % 3 == 1 && m < 12) rot_word(rin, m / 3, rlo, rhi);
        if (m == 11) rot_store(j + 2, rlo, rhi);  // into the buffer QK(j) released
        __builtin_amdgcn_sched_barrier(0);
      }
      const float ps = ps0 + ps1;
      late_bad |= __ballot(ps > p_hi);
      l_run += ps;
      pend = e3;
    } else {
      __builtin_amdgcn_iglp_opt(0);
      qk(kbuf(j + 1), nxt);
      const Ent e3 = ent_of(min(j + 3, n_steps - 1));
      float ps = softmax(cur, pb);
      ref_fix(cur, nxt, pb, ps);
      l_run += ps;
      const RotIn rin = rot_load(pend);  // loaded late: short-lived registers
      pv(vbuf(j), pb);
      rotate(rin, j + 2);
      pend = e3;
    }
  };
  // segment [j, jend): the first tile's scores are in sc_a on entry
  auto segment = [&](int j, int jend, int lo, int hi, Ent& pend) __attribute__((always_inline)) {
    for (; j + 2 <= jend; j += 2) {
      visit(j, sc_a, sc_b, lo, hi, pend);
      visit(j + 1, sc_b, sc_a, lo, hi, pend);
    }
    if (j < jend) visit(j, sc_a, sc_b, lo, hi, pend);
  };

  // ---- prologue: the first view's query operand; K(0), K(1) rotated into
  // their buffers, V(0) in flight
  const bool q_remote = n_r > 0 || REMOTE2;
  load_q_operand(qrow, hl32, q_remote ? rtable : a.table,
                 q_remote && !a.freq_map ? remote_pos(qp, gdiv) : qp, a.q_scale, qop);
  if (CHECK_LATE && tid == 0) s_bad = 0;  // read after the end-of-block barrier
  const int last = n_steps - 1;
  if constexpr (PAGED) {  // the sequence's page list, clamped into the pool
    const int np = min((Lk + (1 << a.page_shift) - 1) >> a.page_shift, kMaxSeqPages);
    for (int i = tid; i < np; i += kPfThreads) {
      const int pg = a.block_table[(size_t)W.b * a.max_pages + i];
      s_pages[i] = pg < 0 ? 0 : (pg >= a.n_pages ? a.n_pages - 1 : pg);
    }
    __syncthreads();
  }
  Ent pend = ent_of(0);
  {
    const Ent e1 = ent_of(min(1, last));
    issue_v(0, 0);
    const RotIn r0 = rot_load(pend), r1 = rot_load(e1);
    rotate(r0, 0);
    rotate(r1, 1);
  }
  __syncthreads();  // the rows of buffer 0 are read by every wave
  pend = ent_of(min(2, last));
  qk(kbuf(0), sc_a);

  if (FUSED && n_r > 0) {
    int lo = 0, hi = 0;
    if (!SAFE) seg1_bounds(lo, hi);
    segment(0, n_r, lo, hi, pend);
    // segment 2 in the base view: its first tile, already rotated to the base
    // view (buffer n_r & 1, not overwritten since), is scored again with the
    // base-rotated query operand
    load_q_operand(qrow, hl32, a.table, qp, a.q_scale, qop);
    qk(kbuf(n_r), sc_a);
  }
  {
    int lo = 0, hi = 0;
    if (!SAFE) seg2_bounds(lo, hi);
    segment(n_r, n_steps, lo, hi, pend);
  }
  wait_vmem();  // the copies past the list's end

  // ---- normalise and write
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (CHECK_LATE) {
    late_bad |= __ballot(row_valid && !(l_tot >= p_lo));
    if (late_bad != 0 && lane == 0) s_bad = 1;
    __syncthreads();
    if (s_bad != 0) {
      if (tid == 0) a.retry_list[atomicAdd(a.retry_count, 1)] = bid;
      return;
    }
  }
  if (row_valid) {
    const float inv = 1.f / l_tot;
    const size_t orow_off = ((row_base + qr) * a.Hq + hd) * kHeadDim;
#pragma unroll
    for (int db = 0; db < 4; ++db) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        f32x4 t;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) t[jj] = acc_o[db][4 * q4 + jj] * inv;
        const int d = 32 * db + 8 * q4 + 4 * hl32;
        if (OUT_F32)
          *(f32x4*)(a.o32 + orow_off + d) = t;
        else
          *(bf16x4*)(a.o + orow_off + d) = __builtin_convertvector(t, bf16x4);
      }
    }
    if (a.lse != nullptr && hl32 == 0)
      a.lse[lse_base + (size_t)hd * a.Lq + qr] = (m_ref + log2f(l_tot)) * 0.69314718055994531f;
  }
}

// ------------------------------------------------------ Eq. (7) merge kernel
// The literal combination of the three window states, per query row:
//   M = max(l_A, l_B, l_C),  W_X = exp(l_X - M),
//   O = (W_A O_A + (W_B O_B - W_C O_C)) / (W_A + (W_B - W_C)),  lse = M + ln(den),
// in fp32 with contraction off.  B and C are subtracted first: for a row whose
// remote-only key set is empty (q <= w0) the two passes are bit-identical and
// their terms cancel exactly.
struct MergeArgs {
  const float* o3;    // O_A, O_B, O_C: [B][L][Hq][128] each, o_stride floats apart
  const float* lse3;  // LSE_A, LSE_B, LSE_C: [B][Hq][L] each, l_stride floats apart
  uint16_t* o;        // bf16 [B][L][Hq][128]
  float* lse;         // optional fp32 [B][Hq][L]
  int L, Hq;
  size_t rows, o_stride, l_stride;
};

// 32 lanes per row (4 channels each), 8 rows per 256-thread workgroup.
__global__ __launch_bounds__(256) void literal_merge_kernel(MergeArgs a) {
#pragma clang fp contract(off)
  const size_t r = (size_t)blockIdx.x * 8 + (threadIdx.x >> 5);
  if (r >= a.rows) return;
  const int c = 4 * (threadIdx.x & 31);
  const int h = (int)(r % a.Hq);
  const size_t bq = r / a.Hq;
  const int qpos = (int)(bq % a.L);
  const size_t b = bq / a.L;
  const size_t li = (b * a.Hq + h) * a.L + qpos;
  const float la = a.lse3[li], lb = a.lse3[li + a.l_stride], lc = a.lse3[li + 2 * a.l_stride];
  const float M = fmaxf(la, fmaxf(lb, lc));
  const float wa = expf(la - M), wb = expf(lb - M), wc = expf(lc - M);
  const float* src = a.o3 + r * kHeadDim + c;
  const f32x4 oa = *(const f32x4*)src;
  const f32x4 ob = *(const f32x4*)(src + a.o_stride);
  const f32x4 oc = *(const f32x4*)(src + 2 * a.o_stride);
  const float den = wa + (wb - wc);
  f32x4 out;
#pragma unroll
  for (int i = 0; i < 4; ++i) out[i] = (wa * oa[i] + (wb * ob[i] - wc * oc[i])) / den;
  *(bf16x4*)(a.o + r * kHeadDim + c) = __builtin_convertvector(out, bf16x4);
  if (a.lse != nullptr && c == 0) a.lse[li] = M + logf(den);
}

// ---------------------------------------------------------------- launchers
// V^T tile images, then the retry counter (256 B) and list (one int per
// workgroup: at most L query blocks per (b, kv head), since BQ = rows / g can
// be as small as 1).  No rotated key is ever stored: K is read raw by the
// attention kernel.
static size_t retry_bytes(long long nwg) { return 256 + (size_t)nwg * sizeof(int); }

static size_t image_bytes(int B, int Hkv, int L) {
  const size_t tiles = (size_t)(L + kPfBK - 1) / kPfBK;
  return (size_t)B * Hkv * tiles * kTileBytes;
}

size_t prefill_workspace_bytes(bool /*bifocal*/, int B, int Hkv, int L) {
  return image_bytes(B, Hkv, L) + retry_bytes((long long)B * Hkv * L);
}

// Literal mode workspace: O_A, O_B, O_C (fp32 [B][L][Hq][128] each), then
// LSE_A, LSE_B, LSE_C (fp32 [B][Hq][L] each), then at the next 256-byte
// boundary the V^T images and the window passes' rerun counters and list,
// laid out as the library scratch.
static size_t round256(size_t x) { return (x + 255) & ~(size_t)255; }
size_t literal_workspace_bytes(int B, int Hq, int Hkv, int L) {
  const size_t rows = (size_t)B * L * Hq;
  return 3 * rows * kHeadDim * sizeof(float) + round256(3 * rows * sizeof(float)) +
         image_bytes(B, Hkv, L) + retry_bytes((long long)B * Hkv * L);
}

// rtable: the remote view's table, nullptr for the aliasing map (then the
// base table is read at f(p)); with freq_map it is read at p.  With
// `retry`, the rerun counter and list follow the images (the prep kernel
// zeroes the counter); without, nothing past the images is touched.
struct Paging {
  const int32_t* block_table;  // nullptr: dense caches
  int max_pages, page_shift, n_pages;
};

static hipError_t launch_prep(const uint16_t* k, const uint16_t* v, const float2* table,
                              const float2* rtable, const uint32_t* table16,
                              const uint32_t* rtable16, int freq_map, int B, int Hkv, int L,
                              int kv_stride, int G, void* images, bool retry, PrefillArgs& a,
                              hipStream_t stream, Paging pg = Paging{nullptr, 0, 0, 0}) {
  a.block_table = pg.block_table;
  a.max_pages = pg.max_pages;
  a.page_shift = pg.page_shift;
  a.n_pages = pg.n_pages;
  const int n_tiles = (L + kPfBK - 1) / kPfBK;
  const size_t img = (size_t)B * Hkv * n_tiles * (kTileBytes / 2);  // bf16 elements of the images
  a.k = k;
  a.kv_stride = kv_stride;
  a.vt = (const uint16_t*)images;
  a.retry_count = retry ? (int*)(a.vt + img) : nullptr;
  a.retry_list = retry ? a.retry_count + 64 : nullptr;
  a.n_tiles = n_tiles;
  a.table = table;
  a.rtable = freq_map ? rtable : table;
  a.table16 = table16;
  a.rtable16 = freq_map ? rtable16 : table16;
  a.freq_map = freq_map;
  a.gdiv = make_fastdiv((uint32_t)G);

  PrepArgs p = {};
  p.v = v;
  p.vt = (uint16_t*)a.vt;
  p.B = B;
  p.Hkv = Hkv;
  p.L = L;
  p.kv_stride = kv_stride;
  p.n_tiles = n_tiles;
  p.retry_count = a.retry_count;
  p.block_table = pg.block_table;
  p.max_pages = pg.max_pages;
  p.page_shift = pg.page_shift;
  p.n_pages = pg.n_pages;
  if ((long long)B * Hkv > 65535) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(vt_prep_kernel, dim3(n_tiles, B * Hkv), dim3(256), 0, stream, p);
  return hipGetLastError();
}

// L: keys of the call; the queries are rows q_start .. q_start + Lq - 1
static void fill_geometry(PrefillArgs& a, int B, int Hq, int Hkv, int L, int q_start, int Lq,
                          float slack) {
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.L = L;
  a.q_start = q_start;
  a.Lq = Lq;
  a.g = Hq / Hkv;
  a.BQ = kPfRows / a.g;
  a.n_qblocks = (Lq + a.BQ - 1) / a.BQ;
  a.q_scale = 1.4426950408889634f / sqrtf((float)kHeadDim);
  a.slack = slack;
}

// The fused and vanilla modes: the fast pass over the grid, then the checked
// pass over the blocks it listed (same grid size; the rest exit at once).
template <int MODE, bool PAGED = false>
static hipError_t launch_fast_then_checked(const PrefillArgs& a, dim3 grid, hipStream_t stream) {
  hipLaunchKernelGGL((prefill_kernel<MODE, false, PAGED>), grid, dim3(kPfThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((prefill_kernel<MODE, true, PAGED>), grid, dim3(kPfThreads), 0, stream, a);
  return hipGetLastError();
}

static hipError_t launch_attn(int mode, const PrefillArgs& a, hipStream_t stream) {
  const long long nwg = (long long)a.n_qblocks * a.B * a.Hkv;
  if (nwg > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  const dim3 grid((unsigned)nwg);
  if (a.block_table != nullptr) {  // paged caches: the chunk entry points only
    if (mode == kModeFused) return launch_fast_then_checked<kModeFused, true>(a, grid, stream);
    if (mode == kModeVanilla) return launch_fast_then_checked<kModeVanilla, true>(a, grid, stream);
    return hipErrorInvalidValue;
  }
  switch (mode) {
    case kModeFused: return launch_fast_then_checked<kModeFused>(a, grid, stream);
    case kModeVanilla: return launch_fast_then_checked<kModeVanilla>(a, grid, stream);
    case kModeWinA: return launch_fast_then_checked<kModeWinA>(a, grid, stream);
    case kModeWinB: return launch_fast_then_checked<kModeWinB>(a, grid, stream);
    case kModeWinC: return launch_fast_then_checked<kModeWinC>(a, grid, stream);
    default: return hipErrorInvalidValue;
  }
}

// Queries at positions q_start .. q_start + Lq - 1 (q, o: [B][Lq][Hq][128],
// lse [B][Hq][Lq]) over keys [0, L) of k, v ([B][kv_stride][Hkv][128]); the
// full prefill is q_start = 0, Lq = kv_stride = L.  ev0 / ev1 (optional) are
// recorded on the stream around the attention kernel.
hipError_t launch_prefill_chunk(bool bifocal, const uint16_t* q, const uint16_t* k,
                                const uint16_t* v, uint16_t* o, float* lse, const float2* table,
                                const float2* rtable, const uint32_t* table16,
                                const uint32_t* rtable16, int freq_map, int B, int Hq, int Hkv,
                                int L, int q_start, int Lq, int kv_stride, int G, int w0,
                                float slack, void* ws, hipStream_t stream, hipEvent_t ev0,
                                hipEvent_t ev1, const int32_t* block_table, int max_pages,
                                int page_shift, int n_pages) {
  PrefillArgs a = {};
  fill_geometry(a, B, Hq, Hkv, L, q_start, Lq, slack);
  hipError_t e = launch_prep(k, v, table, rtable, table16, rtable16, freq_map, B, Hkv, L,
                             kv_stride, G, ws, true, a, stream,
                             Paging{block_table, max_pages, page_shift, n_pages});
  if (e != hipSuccess) return e;
  a.q = q;
  a.o = o;
  a.lse = lse;
  a.w0 = bifocal ? w0 : INT_MAX;
  if (ev0 != nullptr && (e = hipEventRecord(ev0, stream)) != hipSuccess) return e;
  e = launch_attn(bifocal ? kModeFused : kModeVanilla, a, stream);
  if (e == hipSuccess && ev1 != nullptr) e = hipEventRecord(ev1, stream);
  return e;
}

// Eq. (7) taken literally: the three window passes, then the merge.
hipError_t launch_prefill_literal(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                  uint16_t* o, float* lse, const float2* table,
                                  const float2* rtable, const uint32_t* table16,
                                  const uint32_t* rtable16, int freq_map, int B, int Hq, int Hkv,
                                  int L, int G, int w0, float slack, void* ws,
                                  hipStream_t stream) {
  const size_t rows = (size_t)B * L * Hq;
  float* o3 = (float*)ws;
  float* lse3 = o3 + 3 * rows * kHeadDim;
  void* images = (unsigned char*)ws + 3 * rows * kHeadDim * sizeof(float) +
                 round256(3 * rows * sizeof(float));
  PrefillArgs a = {};
  fill_geometry(a, B, Hq, Hkv, L, 0, L, slack);
  // each window runs as the fused call does: a fast pass, then the checked
  // rerun of the blocks it lists.  The passes count their blocks in counters
  // of their own (all zeroed by the prep kernel) and share the list, which
  // each pass's rerun has read before the next pass writes it (one stream).
  hipError_t e = launch_prep(k, v, table, rtable, table16, rtable16, freq_map, B, Hkv, L, L, G,
                             images, true, a, stream);
  if (e != hipSuccess) return e;
  a.q = q;
  int* const counters = a.retry_count;
  const int modes[3] = {kModeWinA, kModeWinB, kModeWinC};
  for (int x = 0; x < 3; ++x) {
    a.o32 = o3 + (size_t)x * rows * kHeadDim;
    a.lse = lse3 + (size_t)x * rows;
    a.w0 = modes[x] == kModeWinB ? INT_MAX : w0;
    a.retry_count = counters + x;
    e = launch_attn(modes[x], a, stream);
    if (e != hipSuccess) return e;
  }
  MergeArgs m;
  m.o3 = o3;
  m.lse3 = lse3;
  m.o = o;
  m.lse = lse;
  m.L = L;
  m.Hq = Hq;
  m.rows = rows;
  m.o_stride = rows * kHeadDim;
  m.l_stride = rows;
  const size_t nblk = (rows + 7) / 8;
  if (nblk > 0x7fffffffULL) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(literal_merge_kernel, dim3((unsigned)nblk), dim3(256), 0, stream, m);
  return hipGetLastError();
}

// ------------------------------------------------- packed (varlen) batches
// Sequence s of a packed batch holds rows cu[s] .. cu[s + 1] - 1 of q, k, v
// and o.  Its bounds are clamped into [0, T] (a non-increasing entry gives an
// empty sequence) and its length to max_len.  The work lists hold one
// (seq0, L, index, tile0) per query block (index = block, last block first)
// and per key tile (index = tile); their sizes nq = ceil(T / BQ) + B and
// nt = ceil(T / 64) + B bound the totals of any well-formed cu.  A sequence
// whose entries would run past either list (possible only for malformed
// cu) gets none: its output rows are left untouched.  Every list entry is
// written exactly once, unused ones as empty (L = 0).
struct PlanArgs {
  const int32_t* cu;
  int B, T, max_len, BQ;
  int4* qwork;
  int4* twork;
  int nq, nt;
};

constexpr int kPlanThreads = 1024;

__global__ __launch_bounds__(kPlanThreads) void varlen_plan_kernel(PlanArgs a) {
  __shared__ long long inc_q[kPlanThreads], inc_t[kPlanThreads];  // inclusive scans
  __shared__ int s_seq0[kPlanThreads], s_len[kPlanThreads];
  const int t = threadIdx.x;
  long long base_q = 0, base_t = 0;  // entries before this chunk of sequences
  for (int c0 = 0; c0 < a.B; c0 += kPlanThreads) {
    const int s = c0 + t;
    int seq0 = 0, len = 0;
    if (s < a.B) {
      seq0 = min(max(a.cu[s], 0), a.T);
      const int seq1 = min(max(a.cu[s + 1], seq0), a.T);
      len = min(seq1 - seq0, a.max_len);
    }
    s_seq0[t] = seq0;
    s_len[t] = len;
    inc_q[t] = (len + a.BQ - 1) / a.BQ;
    inc_t[t] = (len + kPfBK - 1) / kPfBK;
    __syncthreads();
    for (int d = 1; d < kPlanThreads; d <<= 1) {  // Hillis-Steele scan
      const long long xq = t >= d ? inc_q[t - d] : 0;
      const long long xt = t >= d ? inc_t[t - d] : 0;
      __syncthreads();
      inc_q[t] += xq;
      inc_t[t] += xt;
      __syncthreads();
    }
    const long long tot_q = inc_q[kPlanThreads - 1], tot_t = inc_t[kPlanThreads - 1];
    // entry e of this chunk belongs to the first sequence whose inclusive
    // count exceeds e (binary search; sequences without entries are skipped)
    auto owner = [&](const long long* inc, long long e) {
      int lo = 0, hi = kPlanThreads - 1;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (inc[mid] > e) hi = mid; else lo = mid + 1;
      }
      return lo;
    };
    auto fits = [&](int j) {
      return base_q + inc_q[j] <= a.nq && base_t + inc_t[j] <= a.nt;
    };
    for (long long e = t; e < tot_q && base_q + e < a.nq; e += kPlanThreads) {
      const int j = owner(inc_q, e);
      const int nb = (s_len[j] + a.BQ - 1) / a.BQ;
      const long long i = e - (inc_q[j] - nb);
      const long long toff = base_t + inc_t[j] - (s_len[j] + kPfBK - 1) / kPfBK;
      a.qwork[base_q + e] = fits(j) ? int4{s_seq0[j], s_len[j], (int)(nb - 1 - i), (int)toff}
                                    : int4{0, 0, 0, 0};
    }
    for (long long e = t; e < tot_t && base_t + e < a.nt; e += kPlanThreads) {
      const int j = owner(inc_t, e);
      const int nk = (s_len[j] + kPfBK - 1) / kPfBK;
      const long long i = e - (inc_t[j] - nk);
      a.twork[base_t + e] = fits(j) ? int4{s_seq0[j], s_len[j], (int)i, (int)(inc_t[j] - nk + base_t)}
                                    : int4{0, 0, 0, 0};
    }
    base_q += tot_q;
    base_t += tot_t;
    __syncthreads();  // the next chunk reuses the scans
  }
  for (long long e = min(base_q, (long long)a.nq) + t; e < a.nq; e += kPlanThreads)
    a.qwork[e] = int4{0, 0, 0, 0};
  for (long long e = min(base_t, (long long)a.nt) + t; e < a.nt; e += kPlanThreads)
    a.twork[e] = int4{0, 0, 0, 0};
}

static void varlen_sizes(int B, int T, int g, long long* nq, long long* nt) {
  const int BQ = kPfRows / g;
  *nq = ((long long)T + BQ - 1) / BQ + B;
  *nt = ((long long)T + kPfBK - 1) / kPfBK + B;
}

// Scratch of a packed call: the V^T images of nt tiles per kv head (kv head
// h's at h * nt), the query-block and tile work lists, the rerun counter and
// list, then (frequency map only) the per-sequence remote tables, fp32 and
// bf16, one row per token.
static size_t varlen_lists_end(int B, int T, int Hq, int Hkv) {
  long long nq, nt;
  varlen_sizes(B, T, Hq / Hkv, &nq, &nt);
  return (size_t)Hkv * nt * kTileBytes + (size_t)(nq + nt) * sizeof(int4) + retry_bytes(nq * Hkv);
}

size_t prefill_varlen_workspace_bytes(bool bifocal, int B, int T, int Hq, int Hkv, bool freq) {
  (void)bifocal;  // one V^T image set either way
  const size_t base = varlen_lists_end(B, T, Hq, Hkv);
  if (!freq) return base;
  return round256(base) + (size_t)T * kHalf * (sizeof(float2) + sizeof(uint32_t));
}

hipError_t launch_packed_freq_table(const int4* twork, int nt, int w_pre, const double* og,
                                    float2* table, uint32_t* table16, hipStream_t stream);

// Packed batch: q, o [T][Hq][128], k, v [T][Hkv][128], lse [Hq][T] (optional),
// cu: B + 1 device int32.  Each sequence is prefilled as a call with its own
// L, G and positions 0 .. L - 1 (table must cover max_len positions).
hipError_t launch_prefill_varlen(bool bifocal, const uint16_t* q, const uint16_t* k,
                                 const uint16_t* v, uint16_t* o, float* lse, const float2* table,
                                 const uint32_t* table16, const int32_t* cu, int B, int T,
                                 int max_len, int Hq, int Hkv,
                                 int w_pre, int w0, float slack, void* ws, hipStream_t stream,
                                 hipEvent_t ev0, hipEvent_t ev1, const double* freq_og) {
  long long nq, nt;
  varlen_sizes(B, T, Hq / Hkv, &nq, &nt);
  if (nq * Hkv > 0x7fffffffLL || nt > 0x7fffffffLL || Hkv > 65535)
    return hipErrorInvalidConfiguration;
  const size_t img = (size_t)Hkv * nt * (kTileBytes / 2);  // bf16 elements of the V^T images
  PrefillArgs a = {};
  fill_geometry(a, 1, Hq, Hkv, max_len, 0, T, slack);
  a.k = k;
  a.vt = (const uint16_t*)ws;
  int4* qwork = (int4*)((uint16_t*)ws + img);
  int4* twork = qwork + nq;
  a.retry_count = (int*)(twork + nt);
  a.retry_list = a.retry_count + 64;
  a.n_tiles = (int)nt;
  a.table = table;
  a.rtable = table;
  a.table16 = table16;
  a.rtable16 = table16;
  a.freq_map = 0;
  a.gdiv = make_fastdiv(1);
  a.q = q;
  a.o = o;
  a.lse = lse;
  a.w0 = bifocal ? w0 : INT_MAX;
  a.qwork = qwork;
  a.w_pre = w_pre;

  PlanArgs pl;
  pl.cu = cu;
  pl.B = B;
  pl.T = T;
  pl.max_len = max_len;
  pl.BQ = a.BQ;
  pl.qwork = qwork;
  pl.twork = twork;
  pl.nq = (int)nq;
  pl.nt = (int)nt;
  hipLaunchKernelGGL(varlen_plan_kernel, dim3(1), dim3(kPlanThreads), 0, stream, pl);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (bifocal && freq_og != nullptr) {  // each sequence's frequency-map rows, at its own rows
    unsigned char* rt = (unsigned char*)ws + round256(varlen_lists_end(B, T, Hq, Hkv));
    float2* rt32 = (float2*)rt;
    uint32_t* rt16 = (uint32_t*)(rt + (size_t)T * kHalf * sizeof(float2));
    e = launch_packed_freq_table(twork, (int)nt, w_pre, freq_og, rt32, rt16, stream);
    if (e != hipSuccess) return e;
    a.rtable = rt32;
    a.rtable16 = rt16;
    a.freq_map = 1;
    a.rtab_packed = 1;
  }

  PrepArgs p = {};
  p.v = v;
  p.vt = (uint16_t*)a.vt;
  p.B = 1;
  p.Hkv = Hkv;
  p.L = max_len;
  p.kv_stride = T;
  p.n_tiles = (int)nt;
  p.twork = twork;
  p.retry_count = a.retry_count;
  hipLaunchKernelGGL(vt_prep_kernel, dim3((unsigned)nt, Hkv), dim3(256), 0, stream, p);
  if ((e = hipGetLastError()) != hipSuccess) return e;

  if (ev0 != nullptr && (e = hipEventRecord(ev0, stream)) != hipSuccess) return e;
  const dim3 grid((unsigned)(nq * Hkv));
  e = bifocal ? launch_fast_then_checked<kModeFused>(a, grid, stream)
              : launch_fast_then_checked<kModeVanilla>(a, grid, stream);
  if (e == hipSuccess && ev1 != nullptr) e = hipEventRecord(ev1, stream);
  return e;
}

int prefill_rows_per_block() { return kPfRows; }
int prefill_block_q(int g) { return kPfRows / g; }
int prefill_block_k() { return kPfBK; }

}  // namespace jl
