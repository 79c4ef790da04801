// prefill.hip -- fused causal bifocal-RoPE attention, prefill, for gfx950.
//
// Jet-Long (arXiv 2607.07740): a key k <= q is scored with the base rotation
// R(q), R(k) when q - k <= w0 and with the remote rotation R(f(q)), R(f(k)),
// f(x) = floor(x / G), otherwise (Sec. 3, Eq. (1); Sec. 3.1, Eqs. (2)-(3)).
// Raw (pre-RoPE) Q/K are rotated in registers; a key's remote rotation is
// produced while its tile is staged into LDS and is never written to HBM
// (Sec. 3.2: keys stay in base coordinates, the remote view is formed on the
// fly).
//
// Two views, one running state.  For a block of queries the key tiles that
// hold remote pairs are visited first with the remote-rotated query operand,
// then the tiles that hold band pairs with the base-rotated operand; a tile
// straddling the band edge is visited once per view, each visit keeping only
// its own view's elements.  Every visit produces a partial softmax state over
// disjoint keys and is folded into the running fp32 state (m, l, O) with the
// max-shifted, linear-space merge of Sec. 3.3, Eq. (7).  Band keys never enter
// the remote state, so the exclusion window C of Eq. (7) is empty and nothing
// is subtracted.  The vanilla kernel is the same code with only the base view.
//
// Work decomposition (workgroup = 8 wave64s = 256 query rows):
//   rows r of a workgroup are (head hl = r / BQ, position q0 + r % BQ) for the
//   g = Hq/Hkv query heads sharing one kv head (GQA packing), BQ = 256 / g, so
//   one staged K/V tile serves all g heads and its rotation cost is spread
//   over 256 rows.
//   Tiles of 64 keys are double-buffered in LDS: while the waves compute tile
//   t, the raw K/V rows and cos/sin rows of tile t+1 are already in flight to
//   registers; after the compute they are rotated (K) and stored (K, V) into
//   the other buffer, and one barrier closes the step.
//   Each wave computes S^T = K Q^T for its 32 rows with
//   v_mfma_f32_32x32x16_bf16 (a lane owns one query column, so the row
//   maximum is lane-local plus one exchange with lane ^ 32), then
//   O^T += V^T P^T with V^T fed by the transposing LDS read.
//   Softmax runs in the log2 domain with a lazily updated reference maximum
//   m: the MFMA accumulator starts at -m, so scores come out already shifted;
//   m moves (and O, l are rescaled) only when a tile's scores exceed it by more
//   than 2^8, which keeps every exponent <= 2^8 without a per-tile rescale.
#include <climits>
#include <type_traits>

#include "jl_device.h"

namespace jl {

constexpr int kPfThreads = 512;
constexpr int kPfRows = 256;   // query rows per workgroup, 32 per wave
constexpr int kPfBK = 64;      // keys per tile
constexpr int kKStride = 136;  // bf16 per K row in LDS (272 B = 68 dwords: 16 rows read at one
                               // column hit 16 disjoint 4-bank groups)
constexpr int kVStride = 160;  // bf16 per V row in LDS (320 B = 80 dwords: the 4 rows x 64 B of a
                               // transposing read land on disjoint quarters of the 64 banks)
constexpr int kKBuf = kPfBK * kKStride;
constexpr int kVBuf = kPfBK * kVStride;
constexpr float kRescaleLog2 = 8.f;

struct PrefillArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  float* lse;
  const float2* table;  // [positions][64] (cos, sin) of p * omega_i
  int B, Hq, Hkv, L;
  int g, BQ, n_qblocks;
  int w0;        // local window; INT_MAX for the vanilla kernel
  FastDiv gdiv;  // division by G (Eq. (3))
  float q_scale; // log2(e) / sqrt(head_dim): scores come out in log2 units
};

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

// Raw rows of one tile in flight between their global load and their LDS store.
// Thread t stages key t / 8 of the tile, chunk pair c = t % 8: the slices
// d = 8c..8c+7 and their rotate-half partners d + 64.
struct Stage {
  u32x4 klo, khi, vlo, vhi;
  float4 cs[4];  // (cos, sin) of frequencies 8c .. 8c+7 at the key's position
};

template <bool BIFOCAL>
__global__ __launch_bounds__(kPfThreads) void prefill_kernel(PrefillArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sK[2 * kKBuf];
  __shared__ __attribute__((aligned(16))) uint16_t sV[2 * kVBuf];

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int hl32 = lane >> 5;  // which 8-wide half of a 16-wide k slice this lane feeds

  // ---- workgroup -> (b, kv head, q block), longest q blocks first.  When the
  // (b, kv head) groups are a multiple of the 8 XCDs, consecutive work items
  // land on one XCD so a group's K/V tiles stay in that XCD's L2.
  const int n_groups = a.B * a.Hkv;
  const int bid = blockIdx.x;
  int group, qblk;
  if ((n_groups & 7) == 0) {
    const int work = (bid & 7) * (gridDim.x >> 3) + (bid >> 3);
    group = work / a.n_qblocks;
    qblk = a.n_qblocks - 1 - (work - group * a.n_qblocks);
  } else {
    qblk = a.n_qblocks - 1 - bid / n_groups;
    group = bid - (bid / n_groups) * n_groups;
  }
  const int b = group / a.Hkv;
  const int kvh = group - b * a.Hkv;
  const int L = a.L;
  const int w0 = a.w0;
  const int q0 = qblk * a.BQ;
  const int q1 = min(q0 + a.BQ, L) - 1;

  // ---- this lane's query row
  const int row = wave * 32 + (lane & 31);
  const int hl = row / a.BQ;
  const int qpos = q0 + (row - hl * a.BQ);
  const bool row_valid = qpos < L;
  const int qp = row_valid ? qpos : L - 1;
  const int h = kvh * a.g + hl;
  const uint16_t* qrow = a.q + (((size_t)b * L + qp) * a.Hq + h) * kHeadDim;

  // ---- visit list: remote-view tiles [0, n_r), then base-view tiles from kt_l
  const VisitRanges vr = visit_ranges(q0, q1, w0, kPfBK);
  const int n_kt = vr.n_kt;
  const int n_r = BIFOCAL ? vr.n_r : 0;  // tiles holding a remote pair
  const int kt_l = BIFOCAL ? vr.kt_l : 0;  // first tile holding a band pair
  const int n_steps = n_r + (n_kt - kt_l);

  // ---- staging geometry
  const int st_c = tid & 7;
  const int st_key = tid >> 3;
  const size_t kv_row = (size_t)a.Hkv * kHeadDim;
  const uint16_t* kbase = a.k + ((size_t)b * L * a.Hkv + kvh) * kHeadDim + 8 * st_c;
  const uint16_t* vbase = a.v + ((size_t)b * L * a.Hkv + kvh) * kHeadDim + 8 * st_c;

  // raw K/V rows and the cos/sin row of visit j at its view's position; keys
  // past the sequence read row L-1 and are zeroed (only the last tile has any)
  auto issue = [&](int j, Stage& st) {
    const bool remote = j < n_r;
    const int k0 = (remote ? j : kt_l + (j - n_r)) * kPfBK;
    const int key = min(k0 + st_key, L - 1);
    const uint16_t* kr = kbase + (size_t)key * kv_row;
    const uint16_t* vr = vbase + (size_t)key * kv_row;
    st.klo = load16(kr);
    st.khi = load16(kr + kHalf);
    st.vlo = load16(vr);
    st.vhi = load16(vr + kHalf);
    const int pos = remote ? remote_pos(key, a.gdiv) : key;
    const float4* c4 = (const float4*)(a.table + (size_t)pos * kHalf + 8 * st_c);
#pragma unroll
    for (int t = 0; t < 4; ++t) st.cs[t] = c4[t];
    if (k0 + kPfBK > L && k0 + st_key >= L) st.vlo = st.vhi = u32x4{0, 0, 0, 0};
  };
  // rotate the chunk pair and store K and V rows
  auto commit = [&](int buf, const Stage& st) {
    float lo[8], hi[8], ylo[8], yhi[8];
    unpack8(st.klo, lo);
    unpack8(st.khi, hi);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const float4 w = st.cs[t];
      const int i = 2 * t;
      ylo[i] = lo[i] * w.x - hi[i] * w.y;
      yhi[i] = hi[i] * w.x + lo[i] * w.y;
      ylo[i + 1] = lo[i + 1] * w.z - hi[i + 1] * w.w;
      yhi[i + 1] = hi[i + 1] * w.z + lo[i + 1] * w.w;
    }
    uint16_t* kd = sK + buf * kKBuf + st_key * kKStride + 8 * st_c;
    uint16_t* vd = sV + buf * kVBuf + st_key * kVStride + 8 * st_c;
    *(bf16x8*)kd = pack8(ylo);
    *(bf16x8*)(kd + kHalf) = pack8(yhi);
    *(u32x4*)vd = st.vlo;
    *(u32x4*)(vd + kHalf) = st.vhi;
  };

  // ---- query operand of the first view
  bf16x8 qop[8];
  load_q_operand(qrow, hl32, a.table, n_r > 0 ? remote_pos(qp, a.gdiv) : qp, a.q_scale, qop);

  f32x16 acc_o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc_o[i] = f32x16{};
  float m_ref = -INFINITY;  // reference maximum (log2 units), updated lazily
  float l_run = 0.f;

  Stage st;
  issue(0, st);
  commit(0, st);
  __syncthreads();

  const int g16 = lane >> 4;
  const int i16 = lane & 15;
  const int kap_hi = g16 >> 1;

  // one visit: scores of tile j in one view, online softmax, PV; the next
  // visit's rows are loaded meanwhile and staged into the other buffer
  auto step = [&](int j, auto remote_tag) {
    constexpr bool remote = decltype(remote_tag)::value;
    const int k0 = (remote ? j : kt_l + (j - n_r)) * kPfBK;
    const int buf = j & 1;
    if (j + 1 < n_steps) issue(j + 1, st);  // in flight during the QK products
    __builtin_amdgcn_sched_barrier(0);
    // ---- S^T - m for 2 blocks of 32 keys
    const float c_init = m_ref == -INFINITY ? 0.f : -m_ref;
    f32x16 sc[2];
    const uint16_t* kb_lds = sK + buf * kKBuf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int i = 0; i < 16; ++i) sc[kb][i] = c_init;
      const uint16_t* krow = kb_lds + (32 * kb + (lane & 31)) * kKStride + 8 * hl32;
#pragma unroll
      for (int s = 0; s < 8; ++s) sc[kb] = mfma32(*(const bf16x8*)(krow + 16 * s), qop[s], sc[kb]);
    }

    // stage the next visit into the other buffer now, so its registers are free
    // before the softmax and the PV products
    __builtin_amdgcn_sched_barrier(0);
    if (j + 1 < n_steps) commit(buf ^ 1, st);
    __builtin_amdgcn_sched_barrier(0);

    // ---- element masks where the tile is not wholly inside this view
    const bool need_mask = remote ? !(q0 - (k0 + kPfBK - 1) > w0)
                                  : !(q1 - k0 <= w0 && k0 + kPfBK - 1 <= q0);
    if (need_mask) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int diff = qp - (k0 + 32 * kb + 8 * (i >> 2) + 4 * hl32 + (i & 3));
          const bool keep = remote ? diff > w0 : (diff >= 0 && diff <= w0);
          sc[kb][i] = keep ? sc[kb][i] : -INFINITY;
        }
      }
    }

    __builtin_amdgcn_sched_barrier(0);
    // ---- online softmax with a lazily moved reference maximum
    float mt = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mt = fmaxf(mt, sc[kb][i]);
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const bool upd = m_ref == -INFINITY ? mt != -INFINITY : mt > kRescaleLog2;
    float psum = 0.f;
    bf16x8 pb[4];
    if (__ballot(upd) != 0) {
      const float shift = upd ? mt : 0.f;
      const float alpha = fast_exp2(-shift);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          float p[8];
#pragma unroll
          for (int t = 0; t < 8; ++t) {
            p[t] = fast_exp2(sc[kb][8 * hh + t] - shift);
            psum += p[t];
          }
          pb[2 * kb + hh] = pack8(p);
        }
      }
#pragma unroll
      for (int db = 0; db < 4; ++db) acc_o[db] *= alpha;
      l_run = l_run * alpha + psum;
      if (upd) m_ref = m_ref == -INFINITY ? mt : m_ref + mt;
    } else {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          float p[8];
#pragma unroll
          for (int t = 0; t < 8; ++t) {
            p[t] = fast_exp2(sc[kb][8 * hh + t]);
            psum += p[t];
          }
          pb[2 * kb + hh] = pack8(p);
        }
      }
      l_run += psum;
    }


    // ---- O^T += V^T P^T.  k-step ks covers 16 keys; the P^T operand's k index
    // kappa holds key 8 ((kappa % 8) / 4) + 4 (kappa / 8) + kappa % 4 of the
    // step (the S^T accumulator layout), so V^T is read with that permutation:
    // kappa quads {0, 4, 8, 12} start at keys {0, 8, 4, 12}.
    const uint16_t* v_lds = sV + buf * kVBuf;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int key_a = 16 * ks + 4 * kap_hi + (i16 >> 2);
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const int dcol = 32 * db + 16 * (g16 & 1) + 4 * (i16 & 3);
        const i16x4 lo = lds_read_tr4(v_lds + key_a * kVStride + dcol);
        const i16x4 hi = lds_read_tr4(v_lds + (key_a + 8) * kVStride + dcol);
        acc_o[db] = mfma32(concat_tr(lo, hi), pb[ks], acc_o[db]);
      }
    }

    __syncthreads();
  };

  for (int j = 0; j < n_r; ++j) step(j, std::true_type{});
  if (BIFOCAL && n_r > 0) load_q_operand(qrow, hl32, a.table, qp, a.q_scale, qop);
  for (int j = n_r; j < n_steps; ++j) step(j, std::false_type{});

  // ---- normalise and write
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (row_valid) {
    const float inv = 1.f / l_tot;
    uint16_t* orow = a.o + (((size_t)b * L + qpos) * a.Hq + h) * kHeadDim;
#pragma unroll
    for (int db = 0; db < 4; ++db) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        f32x4 t;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) t[jj] = acc_o[db][4 * q4 + jj] * inv;
        *(bf16x4*)(orow + 32 * db + 8 * q4 + 4 * hl32) = __builtin_convertvector(t, bf16x4);
      }
    }
    if (a.lse != nullptr && hl32 == 0)
      a.lse[((size_t)b * a.Hq + h) * L + qpos] = (m_ref + log2f(l_tot)) * 0.69314718055994531f;
  }
}

// ---------------------------------------------------------------- launcher
hipError_t launch_prefill(bool bifocal, const uint16_t* q, const uint16_t* k, const uint16_t* v,
                          uint16_t* o, float* lse, const float2* table, int B, int Hq, int Hkv,
                          int L, int G, int w0, hipStream_t stream) {
  PrefillArgs a;
  a.q = q;
  a.k = k;
  a.v = v;
  a.o = o;
  a.lse = lse;
  a.table = table;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.L = L;
  a.g = Hq / Hkv;
  a.BQ = kPfRows / a.g;
  a.n_qblocks = (L + a.BQ - 1) / a.BQ;
  a.w0 = bifocal ? w0 : INT_MAX;
  a.gdiv = make_fastdiv((uint32_t)G);
  a.q_scale = 1.4426950408889634f / sqrtf((float)kHeadDim);
  const long long nwg = (long long)a.n_qblocks * B * Hkv;
  if (nwg > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  if (bifocal)
    hipLaunchKernelGGL(prefill_kernel<true>, dim3((unsigned)nwg), dim3(kPfThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(prefill_kernel<false>, dim3((unsigned)nwg), dim3(kPfThreads), 0, stream,
                       a);
  return hipGetLastError();
}

int prefill_rows_per_block() { return kPfRows; }
int prefill_block_q(int g) { return kPfRows / g; }
int prefill_block_k() { return kPfBK; }

}  // namespace jl
