// prefill.hip -- fused causal bifocal-RoPE attention, prefill, for gfx950.
//
// Jet-Long (arXiv 2607.07740): a key k <= q is scored with the base rotation
// R(q), R(k) when q - k <= w0 and with the remote rotation R(f(q)), R(f(k)),
// f(x) = floor(x / G), otherwise (Sec. 3, Eq. (1); Sec. 3.1, Eqs. (2)-(3)).
// Raw (pre-RoPE) Q/K are rotated in registers; the remote rotation of a key is
// produced while its tile is staged into LDS and is never written to HBM
// (Sec. 3.2: the cache keeps base-coordinate keys, the remote view is formed
// on the fly).  The local and remote partial softmax states are combined by
// the max-shifted, linear-space merge of Sec. 3.3, Eq. (7), applied tile by
// tile in fp32: each tile contributes the partial state (m_t, l_t, O_t) of its
// keys, the running state is rescaled by exp2(m_old - M) and the tile's by
// exp2(m_t - M), M the larger maximum.  Band keys only ever enter the base
// view and older keys only the remote view, so the exclusion term of Eq. (7)
// (window C) is zero by construction and nothing is subtracted.
//
// Work decomposition (one workgroup = 4 wave64s = 128 query rows):
//   rows r = 0..127 of a workgroup are (head hl = r / BQ, position q0 + r % BQ)
//   for the g = Hq/Hkv query heads that share one kv head (GQA packing), with
//   BQ = 128 / g, so every K/V tile staged in LDS serves all g heads.
//   K/V tiles of BK = 64 keys are loaded coalesced (16 lanes per 256-byte key
//   row), K is rotated to the view(s) the tile needs, and both are stored to
//   LDS.  Each wave computes S^T = K Q^T for its 32 rows with
//   v_mfma_f32_32x32x16_bf16 (lanes own one query column, so the row max/sum
//   of the online softmax is mostly lane-local), then O^T += V^T P^T with the
//   V^T operand read by the transposing LDS read.
//
// Tile classes (q-block x k-tile): SKIP (not visited), LOCAL (base view only),
// REMOTE (remote view only), MIXED (both products, element-wise choice).  Only
// MIXED and diagonal tiles evaluate element masks.
#include "jl_device.h"

namespace jl {

constexpr int kPfThreads = 256;
constexpr int kPfRows = 128;   // query rows per workgroup
constexpr int kPfBK = 64;      // keys per tile
constexpr int kKStride = 136;  // bf16 per K row in LDS (272 B: conflict-free 16-byte row reads)
constexpr int kVStride = 144;  // bf16 per V row in LDS (288 B: conflict-free transposing reads)

struct PrefillArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  float* lse;
  const float2* table;  // [positions][64] (cos, sin) of p * omega_i
  int B, Hq, Hkv, L;
  int g, BQ, n_qblocks;
  int G, w0;
  float q_scale;  // log2(e) / sqrt(head_dim): scores come out in log2 units
};

// Rotate 8 pairs (x_lo, x_hi) at one position and scale; frequencies i0..i0+7.
__device__ inline void rotate_pairs8(const float* lo, const float* hi, const float2* cs,
                                     float scale, float* ylo, float* yhi) {
  const float4* c4 = (const float4*)cs;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    float4 w = c4[t];  // (cos_i, sin_i, cos_{i+1}, sin_{i+1})
    int j = 2 * t;
    ylo[j] = (lo[j] * w.x - hi[j] * w.y) * scale;
    yhi[j] = (hi[j] * w.x + lo[j] * w.y) * scale;
    ylo[j + 1] = (lo[j + 1] * w.z - hi[j + 1] * w.w) * scale;
    yhi[j + 1] = (hi[j + 1] * w.z + lo[j + 1] * w.w) * scale;
  }
}

// Load one query row's operand: 8 k-steps of 8 bf16 (d = 16 s + 8 * half + j),
// rotated to position pos.  Pairs (s, s + 4) are the rotate-half partners.
__device__ inline void load_q_operand(const uint16_t* qrow, int half, const float2* table,
                                      int pos, float scale, bf16x8* out) {
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    int d = 16 * s + 8 * half;
    float lo[8], hi[8], ylo[8], yhi[8];
    unpack8(load16(qrow + d), lo);
    unpack8(load16(qrow + d + kHalf), hi);
    rotate_pairs8(lo, hi, table + (size_t)pos * kHalf + d, scale, ylo, yhi);
    out[s] = pack8(ylo);
    out[s + 4] = pack8(yhi);
  }
}

// Rotate one staged 8-element K chunk.  own = this lane's chunk (d = 8c..8c+7),
// oth = the partner chunk (d +- 64) fetched from lane ^ 8; lanes with c < 8 hold
// the low halves (y = x cos - x' sin), lanes with c >= 8 the high halves
// (y = x cos + x' sin).  Frequencies i = 8 (c mod 8) + j.
__device__ inline bf16x8 rotate_chunk(const float* own, const float* oth, const float2* cs,
                                      float sign) {
  const float4* c4 = (const float4*)cs;
  float y[8];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    float4 w = c4[t];
    y[2 * t] = own[2 * t] * w.x + sign * (oth[2 * t] * w.y);
    y[2 * t + 1] = own[2 * t + 1] * w.z + sign * (oth[2 * t + 1] * w.w);
  }
  return pack8(y);
}

template <bool BIFOCAL>
__global__ __launch_bounds__(kPfThreads) void prefill_kernel(PrefillArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sKb[kPfBK * kKStride];
  __shared__ __attribute__((aligned(16))) uint16_t sKr[BIFOCAL ? kPfBK * kKStride : 8];
  __shared__ __attribute__((aligned(16))) uint16_t sV[kPfBK * kVStride];

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int hl32 = lane >> 5;  // which half of the 16-wide k slice this lane feeds

  // ---- workgroup -> (b, kv head, q block); longest q blocks first.  When the
  // number of (b, kv head) groups is a multiple of the 8 XCDs, consecutive
  // work items land on one XCD so a group's K/V tiles stay in that XCD's L2.
  const int n_groups = a.B * a.Hkv;
  const int nwg = gridDim.x;
  int group, qblk;
  if ((n_groups & 7) == 0) {
    const int bid = blockIdx.x;
    const int work = (bid & 7) * (nwg >> 3) + (bid >> 3);
    group = work / a.n_qblocks;
    qblk = a.n_qblocks - 1 - (work - group * a.n_qblocks);
  } else {
    const int bid = blockIdx.x;
    qblk = a.n_qblocks - 1 - bid / n_groups;
    group = bid - (bid / n_groups) * n_groups;
  }
  const int b = group / a.Hkv;
  const int kvh = group - b * a.Hkv;
  const int L = a.L;
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

  bf16x8 qb[8];
  bf16x8 qr[BIFOCAL ? 8 : 1];
  load_q_operand(qrow, hl32, a.table, qp, a.q_scale, qb);
  if constexpr (BIFOCAL) load_q_operand(qrow, hl32, a.table, remote_pos(qp, a.G), a.q_scale, qr);

  f32x16 acc_o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc_o[i] = f32x16{};
  float m_run = -INFINITY;
  float l_run = 0.f;

  // staging geometry: 16 lanes per key row, chunk c = 8-element slice d = 8c..8c+7
  const int st_c = tid & 15;
  const int st_key = tid >> 4;  // 0..15, plus 16 per pass
  const float st_sign = st_c < 8 ? -1.f : 1.f;
  const int st_freq = 8 * (st_c & 7);
  const size_t kv_row = (size_t)a.Hkv * kHeadDim;
  const uint16_t* kbase = a.k + ((size_t)b * L * a.Hkv + kvh) * kHeadDim;
  const uint16_t* vbase = a.v + ((size_t)b * L * a.Hkv + kvh) * kHeadDim;

  const int n_kt = q1 / kPfBK + 1;
  for (int kt = 0; kt < n_kt; ++kt) {
    const int k0 = kt * kPfBK;
    const int k1 = min(k0 + kPfBK, L) - 1;
    const int cls = BIFOCAL ? tile_class(q0, q1, k0, k1, a.w0) : (int)kLocal;
    const bool need_b = cls != kRemote;
    const bool need_r = BIFOCAL && cls != kLocal;
    // element masks: MIXED tiles, and tiles whose (unclipped) key range
    // reaches past the block's first query -- the diagonal and the ragged end
    const bool need_mask = (cls == kMixed) || (k0 + kPfBK - 1 > q0);

    __syncthreads();  // the previous tile's LDS reads are complete
    // ---- stage: raw K/V rows -> rotated K view(s) and V in LDS
#pragma unroll
    for (int pass = 0; pass < 4; ++pass) {
      const int kl = st_key + 16 * pass;
      const int key = k0 + kl;
      const bool kval = key <= k1;
      const int keyc = kval ? key : k1;
      u32x4 kraw = u32x4{0, 0, 0, 0}, vraw = u32x4{0, 0, 0, 0};
      if (kval) {
        kraw = load16(kbase + (size_t)key * kv_row + 8 * st_c);
        vraw = load16(vbase + (size_t)key * kv_row + 8 * st_c);
      }
      *(u32x4*)(sV + kl * kVStride + 8 * st_c) = vraw;
      const u32x4 kpart = swap_half_row(kraw);
      float own[8], oth[8];
      unpack8(kraw, own);
      unpack8(kpart, oth);
      if (need_b) {
        const float2* cs = a.table + (size_t)keyc * kHalf + st_freq;
        *(bf16x8*)(sKb + kl * kKStride + 8 * st_c) = rotate_chunk(own, oth, cs, st_sign);
      }
      if constexpr (BIFOCAL) {
        if (need_r) {
          const float2* cs = a.table + (size_t)remote_pos(keyc, a.G) * kHalf + st_freq;
          *(bf16x8*)(sKr + kl * kKStride + 8 * st_c) = rotate_chunk(own, oth, cs, st_sign);
        }
      }
    }
    __syncthreads();

    // ---- S^T = K Q^T for this wave's 32 query columns, 2 blocks of 32 keys
    f32x16 sb[2], sr[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      sb[kb] = f32x16{};
      sr[kb] = f32x16{};
      const int krow = 32 * kb + (lane & 31);
      if (need_b) {
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          bf16x8 ka = *(const bf16x8*)(sKb + krow * kKStride + 16 * s + 8 * hl32);
          sb[kb] = mfma32(ka, qb[s], sb[kb]);
        }
      }
      if constexpr (BIFOCAL) {
        if (need_r) {
#pragma unroll
          for (int s = 0; s < 8; ++s) {
            bf16x8 ka = *(const bf16x8*)(sKr + krow * kKStride + 16 * s + 8 * hl32);
            sr[kb] = mfma32(ka, qr[s], sr[kb]);
          }
        }
      }
    }

    // ---- choose the view per element (Eq. (1)) and apply the causal mask
    float sv[2][16];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        float x = need_b ? sb[kb][i] : sr[kb][i];
        if (need_mask) {
          const int key = k0 + 32 * kb + 8 * (i >> 2) + 4 * hl32 + (i & 3);
          const int diff = qp - key;
          if (diff < 0) {
            x = -INFINITY;
          } else if (BIFOCAL && diff > a.w0) {
            x = sr[kb][i];
          } else {
            x = sb[kb][i];
          }
        }
        sv[kb][i] = x;
      }
    }

    // ---- online softmax (log2 domain); the two lanes of a query column
    // (lane, lane ^ 32) hold disjoint key rows and share the running max
    float mt = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mt = fmaxf(mt, sv[kb][i]);
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m_run, mt);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = fast_exp2(m_run - m_use);
    float psum = 0.f;
    bf16x8 pb[4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        float p[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          p[j] = fast_exp2(sv[kb][8 * hh + j] - m_use);
          psum += p[j];
        }
        pb[2 * kb + hh] = pack8(p);
      }
    }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int db = 0; db < 4; ++db) acc_o[db] *= alpha;

    // ---- O^T += V^T P^T.  k-step ks covers 16 keys; the P^T operand's k index
    // kappa maps to key 8 ((kappa % 8) / 4) + 4 (kappa / 8) + kappa % 4 of the
    // step (the accumulator layout of S^T), so the V^T operand is read with the
    // same permutation: quads {0,4,8,12} of kappa start at keys {0,8,4,12}.
    const int g16 = lane >> 4;
    const int i16 = lane & 15;
    const int kap_hi = g16 >> 1;  // 0: kappa 0..7, 1: kappa 8..15
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int key_a = 16 * ks + 4 * kap_hi + (i16 >> 2);  // quad kappa = 8 kap_hi
      const int key_b = key_a + 8;                           // quad kappa = 8 kap_hi + 4
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const int dcol = 32 * db + 16 * (g16 & 1) + 4 * (i16 & 3);
        i16x4 lo = lds_read_tr4(sV + key_a * kVStride + dcol);
        i16x4 hi = lds_read_tr4(sV + key_b * kVStride + dcol);
        acc_o[db] = mfma32(concat_tr(lo, hi), pb[ks], acc_o[db]);
      }
    }
  }

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
        for (int j = 0; j < 4; ++j) t[j] = acc_o[db][4 * q4 + j] * inv;
        bf16x4 ob = __builtin_convertvector(t, bf16x4);
        *(bf16x4*)(orow + 32 * db + 8 * q4 + 4 * hl32) = ob;
      }
    }
    if (a.lse != nullptr && hl32 == 0)
      a.lse[((size_t)b * a.Hq + h) * L + qpos] = (m_run + log2f(l_tot)) * 0.69314718055994531f;
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
  a.G = G;
  a.w0 = w0;
  a.q_scale = 1.4426950408889634f / sqrtf((float)kHeadDim);
  const long long nwg = (long long)a.n_qblocks * B * Hkv;
  if (nwg > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  dim3 grid((unsigned)nwg), block(kPfThreads);
  if (bifocal)
    hipLaunchKernelGGL(prefill_kernel<true>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(prefill_kernel<false>, grid, block, 0, stream, a);
  return hipGetLastError();
}

int prefill_block_q(int g) { return kPfRows / g; }
int prefill_block_k() { return kPfBK; }

}  // namespace jl
