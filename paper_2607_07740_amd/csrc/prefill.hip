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
// Work decomposition: a workgroup is 4 wave64s, one per SIMD, and owns 256
// query rows = (head hl = r / BQ, position q0 + r % BQ) for the g = Hq/Hkv
// query heads sharing one kv head (GQA packing), BQ = 256 / g.  Each wave owns
// 64 rows as two 32-column blocks, so every K and V^T operand it reads from
// LDS feeds two MFMAs and a staged tile's rotation is spread over 256 rows.
// Tiles of 64 keys are double-buffered in LDS; the raw rows of tile t+2 are in
// flight to registers while tile t is computed, and tile t+1 is rotated and
// stored during the last PV products of tile t.
//
// Per tile a wave runs four MFMA groups (v_mfma_f32_32x32x16_bf16): S^T of
// column block 0, S^T of block 1, O^T += V^T P^T for block 0 and for block 1.
// Their VALU partners are laid next to them so one wave's instruction stream
// overlaps matrix and vector work: the softmax of block 0 beside S^T of block
// 1, the softmax of block 1 beside PV of block 0, the next tile's rotation
// beside PV of block 1.  A lane owns one query column of S^T = K Q^T, so the
// row maximum is lane-local plus one exchange with lane ^ 32.
//
// Softmax runs in the log2 domain against a per-row reference maximum m that
// moves only when a tile exceeds it by more than 2^64 (or at the row's first
// key).  -m enters the MFMA itself as one extra k-step (a constant A operand
// with a single 1 against a B operand holding -m), so scores come out already
// shifted and the common path is exp2, sum and convert.  m is kept
// representable in bf16 so that operand is exact.
#include <climits>
#include <type_traits>

#include "jl_device.h"

namespace jl {

constexpr int kPfThreads = 256;  // 4 waves, one per SIMD
constexpr int kPfRows = 256;     // query rows per workgroup: 64 per wave
constexpr int kPfBK = 64;        // keys per tile
constexpr int kKStride = 136;    // bf16 per K row in LDS (272 B = 68 dwords: 16 rows read at one
                                 // column hit 16 disjoint 4-bank groups)
constexpr int kVStride = 160;    // bf16 per V row in LDS (320 B = 80 dwords: the 4 rows x 64 B of
                                 // a transposing read land on disjoint quarters of the 64 banks)
constexpr int kKBuf = kPfBK * kKStride;
constexpr int kVBuf = kPfBK * kVStride;
constexpr float kRescaleLog2 = 64.f;

struct PrefillArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  float* lse;
  const float2* table;  // [positions][64] (cos, sin) of p * omega_i
  int B, Hq, Hkv, L;
  int g, BQ, n_qblocks;
  int w0;         // local window; INT_MAX for the vanilla kernel
  FastDiv gdiv;   // division by G (Eq. (3))
  float q_scale;  // log2(e) / sqrt(head_dim): scores come out in log2 units
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
// Thread t stages keys t / 8 and t / 8 + 32 of the tile, chunk pair c = t % 8:
// the slices d = 8c..8c+7 and their rotate-half partners d + 64.
struct Stage {
  u32x4 klo[2], khi[2], vlo[2], vhi[2];
  float4 cs[2][4];  // (cos, sin) of frequencies 8c .. 8c+7 at each key's position
};

__device__ inline float round_to_bf16(float x) { return (float)(__bf16)x; }

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

  // ---- this lane's two query rows (column blocks qc = 0, 1)
  int qp[2], hd[2];
  bool row_valid[2];
  const uint16_t* qrow[2];
#pragma unroll
  for (int qc = 0; qc < 2; ++qc) {
    const int row = 64 * wave + 32 * qc + (lane & 31);
    const int hl = row / a.BQ;
    const int qpos = q0 + (row - hl * a.BQ);
    row_valid[qc] = qpos < L;
    qp[qc] = row_valid[qc] ? qpos : L - 1;
    hd[qc] = kvh * a.g + hl;
    qrow[qc] = a.q + (((size_t)b * L + qp[qc]) * a.Hq + hd[qc]) * kHeadDim;
  }

  // ---- visit list: remote-view tiles [0, n_r), then base-view tiles from kt_l
  const VisitRanges vr = visit_ranges(q0, q1, w0, kPfBK);
  const int n_kt = vr.n_kt;
  const int n_r = BIFOCAL ? vr.n_r : 0;
  const int kt_l = BIFOCAL ? vr.kt_l : 0;
  const int n_steps = n_r + (n_kt - kt_l);

  // ---- staging geometry
  const int st_c = tid & 7;
  const int st_key = tid >> 3;
  const size_t kv_row = (size_t)a.Hkv * kHeadDim;
  const uint16_t* kbase = a.k + ((size_t)b * L * a.Hkv + kvh) * kHeadDim + 8 * st_c;
  const uint16_t* vbase = a.v + ((size_t)b * L * a.Hkv + kvh) * kHeadDim + 8 * st_c;

  // raw K/V rows and cos/sin rows of visit j at its view's positions; keys
  // past the sequence read row L-1 and their V is zeroed
  auto issue = [&](int j, Stage& st) {
    const bool remote = j < n_r;
    const int k0 = (remote ? j : kt_l + (j - n_r)) * kPfBK;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int key = min(k0 + st_key + 32 * u, L - 1);
      const uint16_t* kr = kbase + (size_t)key * kv_row;
      const uint16_t* vr2 = vbase + (size_t)key * kv_row;
      st.klo[u] = load16(kr);
      st.khi[u] = load16(kr + kHalf);
      st.vlo[u] = load16(vr2);
      st.vhi[u] = load16(vr2 + kHalf);
      const int pos = remote ? remote_pos(key, a.gdiv) : key;
      const float4* c4 = (const float4*)(a.table + (size_t)pos * kHalf + 8 * st_c);
#pragma unroll
      for (int t = 0; t < 4; ++t) st.cs[u][t] = c4[t];
      if (k0 + st_key + 32 * u >= L) st.vlo[u] = st.vhi[u] = u32x4{0, 0, 0, 0};
    }
  };
  // rotate the chunk pairs and store K and V rows into buffer buf
  auto commit = [&](int buf, const Stage& st) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      float lo[8], hi[8], ylo[8], yhi[8];
      unpack8(st.klo[u], lo);
      unpack8(st.khi[u], hi);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const float4 w = st.cs[u][t];
        const int i = 2 * t;
        ylo[i] = lo[i] * w.x - hi[i] * w.y;
        yhi[i] = hi[i] * w.x + lo[i] * w.y;
        ylo[i + 1] = lo[i + 1] * w.z - hi[i + 1] * w.w;
        yhi[i + 1] = hi[i + 1] * w.z + lo[i + 1] * w.w;
      }
      const int kl = st_key + 32 * u;
      uint16_t* kd = sK + buf * kKBuf + kl * kKStride + 8 * st_c;
      uint16_t* vd = sV + buf * kVBuf + kl * kVStride + 8 * st_c;
      *(bf16x8*)kd = pack8(ylo);
      *(bf16x8*)(kd + kHalf) = pack8(yhi);
      *(u32x4*)vd = st.vlo[u];
      *(u32x4*)(vd + kHalf) = st.vhi[u];
    }
  };

  // ---- query operands of the first view, state
  bf16x8 qop[2][8];
#pragma unroll
  for (int qc = 0; qc < 2; ++qc)
    load_q_operand(qrow[qc], hl32, a.table, n_r > 0 ? remote_pos(qp[qc], a.gdiv) : qp[qc],
                   a.q_scale, qop[qc]);

  f32x16 acc_o[2][4];
#pragma unroll
  for (int qc = 0; qc < 2; ++qc)
#pragma unroll
    for (int i = 0; i < 4; ++i) acc_o[qc][i] = f32x16{};
  float m_ref[2] = {-INFINITY, -INFINITY};  // reference maximum (log2 units), bf16-exact
  float l_run[2] = {0.f, 0.f};
  // extra k-step operands adding -m to every score of a column: A holds a single
  // 1 (row k = 0 of the step, lanes 0..31), B holds -m in the same k row
  bf16x8 a_one = bf16x8{};
  if (hl32 == 0) a_one[0] = (__bf16)1.0f;
  bf16x8 b_off[2] = {bf16x8{}, bf16x8{}};

  const int g16 = lane >> 4;
  const int i16 = lane & 15;
  const int kap_hi = g16 >> 1;

  Stage st;
  issue(0, st);
  commit(0, st);
  if (n_steps > 1) issue(1, st);

  // S^T - m for column block qc: 2 blocks of 32 keys, 8 k-steps + the offset step
  auto qk = [&](int qc, int buf, f32x16* sc) {
    const uint16_t* kb_lds = sK + buf * kKBuf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      sc[kb] = mfma32(a_one, b_off[qc], f32x16{});
      const uint16_t* krow = kb_lds + (32 * kb + (lane & 31)) * kKStride + 8 * hl32;
#pragma unroll
      for (int s = 0; s < 8; ++s) sc[kb] = mfma32(*(const bf16x8*)(krow + 16 * s), qop[qc][s], sc[kb]);
    }
  };

  // element masks where the tile is not wholly inside the visit's view
  auto mask = [&](int qc, int k0, bool remote, f32x16* sc) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int diff = qp[qc] - (k0 + 32 * kb + 8 * (i >> 2) + 4 * hl32 + (i & 3));
        const bool keep = remote ? diff > w0 : (diff >= 0 && diff <= w0);
        sc[kb][i] = keep ? sc[kb][i] : -INFINITY;
      }
    }
  };

  // exp2 of the shifted scores; moves the reference maximum when needed
  auto softmax = [&](int qc, f32x16* sc, bf16x8* pb) {
    float mt = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mt = fmaxf(mt, sc[kb][i]);
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    float psum = 0.f;
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
    const bool upd = m_ref[qc] == -INFINITY ? mt != -INFINITY : mt > kRescaleLog2;
    if (__ballot(upd) != 0) {  // rare: the row's first keys or a large jump
      const float m_old = m_ref[qc] == -INFINITY ? 0.f : m_ref[qc];
      const float m_new = upd ? round_to_bf16(m_old + mt) : m_old;
      const float shift = m_new - m_old;
      psum = 0.f;
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
      const float alpha = fast_exp2(-shift);
#pragma unroll
      for (int db = 0; db < 4; ++db) acc_o[qc][db] *= alpha;
      l_run[qc] *= alpha;
      if (upd) {
        m_ref[qc] = m_new;
        if (hl32 == 0) b_off[qc][0] = (__bf16)(-m_new);
      }
    }
    l_run[qc] += psum;
  };

  // O^T += V^T P^T for column block qc.  k-step ks covers 16 keys; the P^T
  // operand's k index kappa holds key 8 ((kappa % 8) / 4) + 4 (kappa / 8) +
  // kappa % 4 of the step (the S^T accumulator layout), so V^T is read with
  // that permutation: kappa quads {0, 4, 8, 12} start at keys {0, 8, 4, 12}.
  auto pv = [&](int qc, int buf, const bf16x8* pb) {
    const uint16_t* v_lds = sV + buf * kVBuf;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int key_a = 16 * ks + 4 * kap_hi + (i16 >> 2);
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const int dcol = 32 * db + 16 * (g16 & 1) + 4 * (i16 & 3);
        const i16x4 lo = lds_read_tr4(v_lds + key_a * kVStride + dcol);
        const i16x4 hi = lds_read_tr4(v_lds + (key_a + 8) * kVStride + dcol);
        acc_o[qc][db] = mfma32(concat_tr(lo, hi), pb[ks], acc_o[qc][db]);
      }
    }
  };

  // one visit of tile j in one view
  auto step = [&](int j, auto remote_tag) {
    constexpr bool remote = decltype(remote_tag)::value;
    const int k0 = (remote ? j : kt_l + (j - n_r)) * kPfBK;
    const int buf = j & 1;
    const bool need_mask = remote ? !(q0 - (k0 + kPfBK - 1) > w0)
                                  : !(q1 - k0 <= w0 && k0 + kPfBK - 1 <= q0);
    __syncthreads();  // tile j is staged; the other buffer is free

    f32x16 sc0[2], sc1[2];
    bf16x8 pb0[4], pb1[4];
    qk(0, buf, sc0);
    if (need_mask) mask(0, k0, remote, sc0);
    __builtin_amdgcn_sched_barrier(0);
    qk(1, buf, sc1);
    __builtin_amdgcn_sched_barrier(0);
    softmax(0, sc0, pb0);
    if (need_mask) mask(1, k0, remote, sc1);
    __builtin_amdgcn_sched_barrier(0);
    pv(0, buf, pb0);
    __builtin_amdgcn_sched_barrier(0);
    softmax(1, sc1, pb1);
    __builtin_amdgcn_sched_barrier(0);
    pv(1, buf, pb1);
    __builtin_amdgcn_sched_barrier(0);
    if (j + 1 < n_steps) commit(buf ^ 1, st);
    __builtin_amdgcn_sched_barrier(0);
    if (j + 2 < n_steps) issue(j + 2, st);
  };

  for (int j = 0; j < n_r; ++j) step(j, std::true_type{});
  if (BIFOCAL && n_r > 0) {
#pragma unroll
    for (int qc = 0; qc < 2; ++qc) load_q_operand(qrow[qc], hl32, a.table, qp[qc], a.q_scale, qop[qc]);
  }
  for (int j = n_r; j < n_steps; ++j) step(j, std::false_type{});

  // ---- normalise and write
#pragma unroll
  for (int qc = 0; qc < 2; ++qc) {
    const float l_tot = l_run[qc] + __shfl_xor(l_run[qc], 32);
    if (row_valid[qc]) {
      const float inv = 1.f / l_tot;
      uint16_t* orow = a.o + (((size_t)b * L + qp[qc]) * a.Hq + hd[qc]) * kHeadDim;
#pragma unroll
      for (int db = 0; db < 4; ++db) {
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          f32x4 t;
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) t[jj] = acc_o[qc][db][4 * q4 + jj] * inv;
          *(bf16x4*)(orow + 32 * db + 8 * q4 + 4 * hl32) = __builtin_convertvector(t, bf16x4);
        }
      }
      if (a.lse != nullptr && hl32 == 0)
        a.lse[((size_t)b * a.Hq + hd[qc]) * L + qp[qc]] =
            (m_ref[qc] + log2f(l_tot)) * 0.69314718055994531f;
    }
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
