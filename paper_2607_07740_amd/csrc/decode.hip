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

constexpr int kDecWaves = 8;  // kv heads per workgroup, one wave each
constexpr int kDecThreads = 64 * kDecWaves;
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
  int chunk, n_split, n_hgroups;
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

// Raw K/V of 32 keys in flight: K in the MFMA A-operand layout (lane holds key
// i16 + 16 hh at d = 32 s + 8 g4 .. +7), V as 16-byte row slices (key 4 r + g4,
// d = 8 i16 .. +7).
struct DecRaw {
  u32x4 k[2][4];
  u32x4 v[8];
  float4 cs[2][2][4];  // cos/sin of each key's view position, frequencies 32 s + 8 g4 .. +7
};

template <bool BIFOCAL>
__global__ __launch_bounds__(kDecThreads, 1) void decode_split_kernel(DecodeArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sV[kDecWaves * kDecWaveKeys * kDecVStride];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int i16 = lane & 15;
  const int g4 = lane >> 4;

  // workgroup = (b, group of up to 8 kv heads, key chunk); wave = one kv head,
  // so the workgroup reads each key's contiguous heads together
  const int bid = blockIdx.x;
  const int split = bid % a.n_split;
  const int t = bid / a.n_split;
  const int hgroup = t % a.n_hgroups;
  const int b = t / a.n_hgroups;
  const int kvh = hgroup * kDecWaves + wave;
  if (kvh >= a.Hkv) return;  // uniform over the wave; no block-level barrier follows
  const int kv_len = clamp_len(a.kv_lens[b], a.max_len);
  const int c0 = split * a.chunk;
  if (c0 >= kv_len) return;
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

  uint16_t* sVw = sV + wave * kDecWaveKeys * kDecVStride;  // this wave's V staging rows
  const size_t kv_row = (size_t)a.Hkv * kHeadDim;
  const uint16_t* kbase = a.kc + ((size_t)b * a.max_len * a.Hkv + kvh) * kHeadDim;
  const uint16_t* vbase = a.vc + ((size_t)b * a.max_len * a.Hkv + kvh) * kHeadDim;

  // keys past the chunk read row c1 - 1 (inside the sequence) and are masked;
  // each key's cos/sin row is the one of the view its distance selects (Eq. (1))
  auto load_raw = [&](int kb0, DecRaw& r) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int keyc = min(kb0 + 16 * hh + i16, c1 - 1);
      const uint16_t* row = kbase + (size_t)keyc * kv_row + 8 * g4;
#pragma unroll
      for (int s = 0; s < 4; ++s) r.k[hh][s] = load16(row + 32 * s);
      int pos = keyc;
      if (BIFOCAL && qpos - keyc > a.w0) pos = remote_pos(keyc, gdiv);
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const float4* c4 = (const float4*)(a.table + (size_t)pos * kHalf + 32 * s + 8 * g4);
#pragma unroll
        for (int t4 = 0; t4 < 4; ++t4) r.cs[hh][s][t4] = c4[t4];
      }
    }
#pragma unroll
    for (int rr = 0; rr < 8; ++rr)
      r.v[rr] = load16(vbase + (size_t)min(kb0 + 4 * rr + g4, c1 - 1) * kv_row + 8 * i16);
  };

  auto process = [&](int kb0, const DecRaw& r) {
    // V rows -> this wave's LDS slice
#pragma unroll
    for (int rr = 0; rr < 8; ++rr) *(u32x4*)(sVw + (4 * rr + g4) * kDecVStride + 8 * i16) = r.v[rr];

    // each key rotated once, to the position its view selects (Eq. (1))
    bf16x8 ka[2][4];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int s = 0; s < 2; ++s)
        rotate8(r.k[hh][s], r.k[hh][s + 2], (const float2*)r.cs[hh][s], 1.f, ka[hh][s],
                ka[hh][s + 2]);

    // S^T (16 keys x 16 columns per block)
    f32x4 sc[2];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      sc[hh] = f32x4{};
#pragma unroll
      for (int s = 0; s < 4; ++s) sc[hh] = mfma16(ka[hh][s], qop[s], sc[hh]);
    }

    // each column keeps only the keys of its own view
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
      const i16x4 v0 = lds_read_tr4(sVw + (4 * g4 + (i16 >> 2)) * kDecVStride + dcol);
      const i16x4 v1 = lds_read_tr4(sVw + (16 + 4 * g4 + (i16 >> 2)) * kDecVStride + dcol);
      acc_o[db] = mfma16(concat_tr(v0, v1), pb, acc_o[db]);
    }
  };

  // ---- stream the chunk, 32 keys per step; the other waves of the workgroup
  // stream the neighbouring heads of the same keys
  for (int kb0 = c0; kb0 < c1; kb0 += kDecWaveKeys) {
    DecRaw r;
    load_raw(kb0, r);
    process(kb0, r);
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
  if (writer && g4 == 0) *(f32x4*)out = f32x4{m_own, W_own * l_own + W_oth * l_oth, 0.f, 0.f};
}

// Final merge over the splits of one head (Eq. (7) weights exp2(m - M)):
// O = sum W O~ / sum W l.  Thread t accumulates output slice t % 32 (4
// channels) over splits t / 32, t / 32 + 8, ...; partial sums meet in LDS.
__global__ __launch_bounds__(256) void decode_reduce_kernel(DecodeArgs a, uint16_t* o) {
  __shared__ float sMax[4];
  __shared__ __attribute__((aligned(16))) float sAcc[8][kHeadDim];
  __shared__ float sDen[8];
  const int bh = blockIdx.x;
  const int b = bh / a.Hq;
  const int tid = threadIdx.x;
  const int kv_len = clamp_len(a.kv_lens[b], a.max_len);
  const int ns = (kv_len + a.chunk - 1) / a.chunk;
  const float* base = a.ws + (size_t)bh * a.n_split * kStateFloats;

  float M = -INFINITY;
  for (int s = tid; s < ns; s += 256) M = fmaxf(M, base[(size_t)s * kStateFloats]);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) M = fmaxf(M, __shfl_xor(M, off));
  if ((tid & 63) == 0) sMax[tid >> 6] = M;
  __syncthreads();
  M = fmaxf(fmaxf(sMax[0], sMax[1]), fmaxf(sMax[2], sMax[3]));

  const int c = tid & 31;
  const int grp = tid >> 5;
  f32x4 acc = f32x4{};
  float den = 0.f;
#pragma unroll 4
  for (int s = grp; s < ns; s += 8) {
    const float* stt = base + (size_t)s * kStateFloats;
    const float m = stt[0];
    const float w = m == -INFINITY ? 0.f : fast_exp2(m - M);
    den += w * stt[1];
    acc += w * *(const f32x4*)(stt + 4 + 4 * c);
  }
  *(f32x4*)&sAcc[grp][4 * c] = acc;
  if (c == 0) sDen[grp] = den;
  __syncthreads();
  if (tid < kHeadDim) {
    float num = 0.f, dsum = 0.f;
#pragma unroll
    for (int g2 = 0; g2 < 8; ++g2) {
      num += sAcc[g2][tid];
      dsum += sDen[g2];
    }
    const __bf16 r = (__bf16)(num / dsum);
    o[(size_t)bh * kHeadDim + tid] = __builtin_bit_cast(uint16_t, r);
  }
}

// ---------------------------------------------------------------- launcher
void decode_geometry(int B, int Hkv, int max_len, int* chunk, int* n_split) {
  // about one 8-wave workgroup per CU (256 CUs): enough waves to stream at
  // full bandwidth while keeping few split states for the reduce; chunks are
  // multiples of one 32-key step
  const long long groups = (long long)B * ((Hkv + kDecWaves - 1) / kDecWaves);
  const long long want = (256 + groups - 1) / groups;
  long long ch = ((long long)max_len + want - 1) / want;
  ch = (ch + kDecWaveKeys - 1) / kDecWaveKeys * kDecWaveKeys;
  if (ch < 128) ch = 128;
  *chunk = (int)ch;
  *n_split = (int)((max_len + ch - 1) / ch);
}

size_t decode_workspace_bytes(int B, int Hq, int Hkv, int max_len) {
  int chunk, n_split, n_hgroups;
  decode_geometry(B, Hkv, max_len, &chunk, &n_split);
  return (size_t)B * Hq * n_split * kStateFloats * sizeof(float);
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
  a.n_hgroups = (Hkv + kDecWaves - 1) / kDecWaves;
  a.w_pre = w_pre;
  a.w0 = w0;
  a.q_scale = 1.4426950408889634f / sqrtf((float)kHeadDim);
  const long long nwg = (long long)a.n_split * a.n_hgroups * B;
  if (nwg > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  if (bifocal) {
    hipLaunchKernelGGL(decode_split_kernel<true>, dim3((unsigned)nwg), dim3(kDecThreads), 0,
                       stream, a);
    hipLaunchKernelGGL(decode_reduce_kernel, dim3(B * Hq), dim3(256), 0, stream, a, o);
  } else {
    hipLaunchKernelGGL(decode_split_kernel<false>, dim3((unsigned)nwg), dim3(kDecThreads), 0,
                       stream, a);
    hipLaunchKernelGGL(decode_reduce_kernel, dim3(B * Hq), dim3(256), 0, stream, a, o);
  }
  return hipGetLastError();
}

}  // namespace jl
