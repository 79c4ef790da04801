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
// Split-K: workgroup (b, kv head, split) streams CH keys of one kv head.  The
// g query heads of the group are rotated twice (base and remote) and placed
// in the 16 columns of a v_mfma_f32_16x16x32_bf16 B operand: columns 0..7 hold
// the base-rotated heads, 8..15 the remote-rotated ones.  Each key is rotated
// once, to the view its distance selects (Eq. (1)), and scored against both
// column groups; a column keeps only keys of its own view, so every column is
// the partial softmax state (m, l, O) of one (head, view) pair: the local
// window state and the remote-only state of Sec. 3.3.  The reduce kernel
// merges all (split, view) states of a head with the max-shifted,
// linear-space rule of Eq. (7) in fp32.
#include "jl_device.h"

namespace jl {

constexpr int kDecThreads = 256;
constexpr int kDecWaveKeys = 32;
constexpr int kDecVStride = 144;     // bf16 per staged V row (transposing reads)
constexpr int kStateFloats = 132;    // m, l, 2 pad, O[128]

struct DecodeArgs {
  const uint16_t* q;
  const uint16_t* kc;
  const uint16_t* vc;
  const int32_t* kv_lens;
  float* ws;
  const float2* table;
  int B, Hq, Hkv, g, max_len;
  int chunk, n_split;
  int w_pre, w0;
  float q_scale;
};

__device__ inline int clamp_len(int n, int max_len) { return n < 1 ? 1 : (n > max_len ? max_len : n); }

// Rotate an 8-element pair of slices (d, d + 64) to the position whose table
// row starts at cs (frequencies d..d+7), optional scale.
__device__ inline void rotate8(const u32x4 rlo, const u32x4 rhi, const float2* cs, float scale,
                               bf16x8& olo, bf16x8& ohi) {
  float lo[8], hi[8], ylo[8], yhi[8];
  unpack8(rlo, lo);
  unpack8(rhi, hi);
  const float4* c4 = (const float4*)cs;
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

template <bool BIFOCAL>
__global__ __launch_bounds__(kDecThreads) void decode_split_kernel(DecodeArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sV[4 * kDecWaveKeys * kDecVStride];

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int i16 = lane & 15;
  const int g4 = lane >> 4;

  const int bid = blockIdx.x;
  const int split = bid % a.n_split;
  const int t = bid / a.n_split;
  const int kvh = t % a.Hkv;
  const int b = t / a.Hkv;
  const int kv_len = clamp_len(a.kv_lens[b], a.max_len);
  const int c0 = split * a.chunk;
  if (c0 >= kv_len) return;  // uniform over the workgroup
  const int c1 = min(c0 + a.chunk, kv_len);
  const int G = BIFOCAL ? group_size(kv_len, a.w_pre) : 1;
  const FastDiv gdiv = make_fastdiv((uint32_t)G);
  const int qpos = kv_len - 1;

  // ---- query operand: column col = (view, head) with view = col / 8
  const int col = i16;
  const int view = col >> 3;
  const int hj = col & 7;
  const bool col_on = hj < a.g && (BIFOCAL || view == 0);
  bf16x8 qop[4];
  if (col_on) {
    const uint16_t* qrow = a.q + ((size_t)b * a.Hq + kvh * a.g + hj) * kHeadDim;
    const int pos = view ? remote_pos(qpos, gdiv) : qpos;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int d = 32 * s + 8 * g4;
      rotate8(load16(qrow + d), load16(qrow + d + kHalf), a.table + (size_t)pos * kHalf + d,
              a.q_scale, qop[s], qop[s + 2]);
    }
  } else {
#pragma unroll
    for (int s = 0; s < 4; ++s) qop[s] = bf16x8{};
  }

  f32x4 acc_o[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc_o[i] = f32x4{};
  float m_run = -INFINITY, l_run = 0.f;

  uint16_t* sVw = sV + wave * kDecWaveKeys * kDecVStride;
  const size_t kv_row = (size_t)a.Hkv * kHeadDim;
  const uint16_t* kbase = a.kc + ((size_t)b * a.max_len * a.Hkv + kvh) * kHeadDim;
  const uint16_t* vbase = a.vc + ((size_t)b * a.max_len * a.Hkv + kvh) * kHeadDim;

  for (int it = 0;; ++it) {
    const int kb0 = c0 + kDecWaveKeys * (wave + 4 * it);
    if (kb0 >= c1) break;  // uniform over the wave

    // V rows of the 32 keys -> this wave's LDS slice (16 lanes per 256-byte row)
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int kl = 4 * r + g4;
      const int key = kb0 + kl;
      u32x4 vraw = u32x4{0, 0, 0, 0};
      if (key < c1) vraw = load16(vbase + (size_t)key * kv_row + 8 * i16);
      *(u32x4*)(sVw + kl * kDecVStride + 8 * i16) = vraw;
    }

    // K operand: 2 blocks of 16 keys, lane holds key i16 at d = 32 s + 8 g4 + j;
    // each key rotated once, to the position its view selects
    bf16x8 ka[2][4];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int key = kb0 + 16 * hh + i16;
      const bool kval = key < c1;
      const int keyc = kval ? key : c1 - 1;
      int pos = keyc;
      if (BIFOCAL && qpos - keyc > a.w0) pos = remote_pos(keyc, gdiv);
      const uint16_t* krow = kbase + (size_t)keyc * kv_row;
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const int d = 32 * s + 8 * g4;
        u32x4 rlo = u32x4{0, 0, 0, 0}, rhi = u32x4{0, 0, 0, 0};
        if (kval) {
          rlo = load16(krow + d);
          rhi = load16(krow + d + kHalf);
        }
        rotate8(rlo, rhi, a.table + (size_t)pos * kHalf + d, 1.f, ka[hh][s], ka[hh][s + 2]);
      }
    }

    // S^T (16 keys x 16 columns per block)
    f32x4 sc[2];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      sc[hh] = f32x4{};
#pragma unroll
      for (int s = 0; s < 4; ++s) sc[hh] = mfma16(ka[hh][s], qop[s], sc[hh]);
    }

    // each column keeps only the keys of its own view (Eq. (1))
    float sv[8];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = kb0 + 16 * hh + 4 * g4 + i;
        bool ok = col_on && key < c1;
        if (BIFOCAL) {
          const bool local = qpos - key <= a.w0;
          ok = ok && (view == 0 ? local : !local);
        }
        sv[4 * hh + i] = ok ? sc[hh][i] : -INFINITY;
      }
    }

    // online softmax per column (the 4 lanes i16, i16+16, i16+32, i16+48)
    float mt = -INFINITY;
#pragma unroll
    for (int j = 0; j < 8; ++j) mt = fmaxf(mt, sv[j]);
    mt = fmaxf(mt, __shfl_xor(mt, 16));
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m_run, mt);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = fast_exp2(m_run - m_use);
    float p[8], psum = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      p[j] = fast_exp2(sv[j] - m_use);
      psum += p[j];
    }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int db = 0; db < 8; ++db) acc_o[db] *= alpha;
    // P^T operand: k index kappa = 8 g4 + j holds key 16 (j / 4) + 4 g4 + j % 4
    const bf16x8 pb = pack8(p);

    // O^T += V^T P^T; V^T read transposed: quad t of this lane group starts at
    // key 16 t + 4 g4
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      const int dcol = 16 * db + 4 * (i16 & 3);
      i16x4 v0 = lds_read_tr4(sVw + (4 * g4 + (i16 >> 2)) * kDecVStride + dcol);
      i16x4 v1 = lds_read_tr4(sVw + (16 + 4 * g4 + (i16 >> 2)) * kDecVStride + dcol);
      acc_o[db] = mfma16(concat_tr(v0, v1), pb, acc_o[db]);
    }
  }

  // ---- merge the 4 waves' states per column, write one state per (head, view)
  float l_tot = l_run + __shfl_xor(l_run, 16);
  l_tot += __shfl_xor(l_tot, 32);
  __syncthreads();
  float* st = (float*)sV;  // [wave][col][kStateFloats] (fits in the V staging area)
  float* mine = st + (wave * 16 + col) * kStateFloats;
  if (g4 == 0) {
    mine[0] = m_run;
    mine[1] = l_tot;
  }
#pragma unroll
  for (int db = 0; db < 8; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) mine[4 + 16 * db + 4 * g4 + i] = acc_o[db][i];
  __syncthreads();

  const int c = tid >> 4;    // column
  const int part = tid & 15; // 8 output channels each
  const int view_c = c >> 3, hj_c = c & 7;
  if (hj_c < a.g && (BIFOCAL || view_c == 0)) {
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, st[(w * 16 + c) * kStateFloats]);
    float W[4];
    float l_sum = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float mw = st[(w * 16 + c) * kStateFloats];
      W[w] = (M == -INFINITY) ? 0.f : fast_exp2(mw - M);
      l_sum += W[w] * st[(w * 16 + c) * kStateFloats + 1];
    }
    const int h = kvh * a.g + hj_c;
    float* out = a.ws + ((((size_t)b * a.Hq + h) * a.n_split + split) * 2 + view_c) * kStateFloats;
    if (part == 0) {
      out[0] = M;
      out[1] = l_sum;
      out[2] = 0.f;
      out[3] = 0.f;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int d = 8 * part + j;
      float acc = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) acc += W[w] * st[(w * 16 + c) * kStateFloats + 4 + d];
      out[4 + d] = acc;
    }
  }
}

// Eq. (7) over all (split, view) states of one head: M = max m, W = exp2(m - M),
// O = sum W O~ / sum W l (the exclusion window is empty: band keys never enter
// the remote states).
template <bool BIFOCAL>
__global__ __launch_bounds__(128) void decode_reduce_kernel(DecodeArgs a, uint16_t* o) {
  const int bh = blockIdx.x;
  const int b = bh / a.Hq;
  const int d = threadIdx.x;
  const int kv_len = clamp_len(a.kv_lens[b], a.max_len);
  const int ns = (kv_len + a.chunk - 1) / a.chunk;
  const int nv = BIFOCAL ? 2 : 1;
  const float* base = a.ws + (size_t)bh * a.n_split * 2 * kStateFloats;
  float M = -INFINITY;
  for (int s = 0; s < ns; ++s)
    for (int v = 0; v < nv; ++v) M = fmaxf(M, base[(s * 2 + v) * kStateFloats]);
  float num = 0.f, den = 0.f;
  for (int s = 0; s < ns; ++s) {
    for (int v = 0; v < nv; ++v) {
      const float* stt = base + (s * 2 + v) * kStateFloats;
      const float m = stt[0];
      const float w = m == -INFINITY ? 0.f : fast_exp2(m - M);
      num += w * stt[4 + d];
      den += w * stt[1];
    }
  }
  const __bf16 r = (__bf16)(num / den);
  o[(size_t)bh * kHeadDim + d] = __builtin_bit_cast(uint16_t, r);
}

// ---------------------------------------------------------------- launcher
void decode_geometry(int B, int Hkv, int max_len, int* chunk, int* n_split) {
  // aim for ~1024 workgroups over the chip; chunks are multiples of 128 keys
  // (4 waves x 32 keys)
  long long groups = (long long)B * Hkv;
  long long want = (1024 + groups - 1) / groups;
  long long ch = ((long long)max_len + want - 1) / want;
  ch = (ch + 127) / 128 * 128;
  if (ch < 128) ch = 128;
  *chunk = (int)ch;
  *n_split = (int)((max_len + ch - 1) / ch);
}

size_t decode_workspace_bytes(int B, int Hq, int Hkv, int max_len) {
  int chunk, n_split;
  decode_geometry(B, Hkv, max_len, &chunk, &n_split);
  return (size_t)B * Hq * n_split * 2 * kStateFloats * sizeof(float);
}

hipError_t launch_decode(bool bifocal, const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                         const int32_t* kv_lens, int max_len, uint16_t* o, const float2* table,
                         int B, int Hq, int Hkv, int w_pre, int w0, float* ws,
                         hipStream_t stream) {
  DecodeArgs a;
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
  decode_geometry(B, Hkv, max_len, &a.chunk, &a.n_split);
  a.w_pre = w_pre;
  a.w0 = w0;
  a.q_scale = 1.4426950408889634f / sqrtf((float)kHeadDim);
  const long long nwg = (long long)a.n_split * Hkv * B;
  if (nwg > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  if (bifocal) {
    hipLaunchKernelGGL(decode_split_kernel<true>, dim3((unsigned)nwg), dim3(kDecThreads), 0,
                       stream, a);
    hipLaunchKernelGGL(decode_reduce_kernel<true>, dim3(B * Hq), dim3(128), 0, stream, a, o);
  } else {
    hipLaunchKernelGGL(decode_split_kernel<false>, dim3((unsigned)nwg), dim3(kDecThreads), 0,
                       stream, a);
    hipLaunchKernelGGL(decode_reduce_kernel<false>, dim3(B * Hq), dim3(128), 0, stream, a, o);
  }
  return hipGetLastError();
}

}  // namespace jl
