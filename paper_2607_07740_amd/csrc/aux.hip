// aux.hip -- RoPE cos/sin tables and the debug views of the device schedule.
#include "jl_device.h"

namespace jl {

struct Omega {
  double w[kHalf];  // omega_i = theta^(-2i/d), computed on the host in fp64
};

// Round an fp64 value to bf16 with one correct round-to-nearest-even step:
// rounding to fp32 toward zero and setting the last bit when inexact (round
// to odd) keeps enough information for the second rounding to be exact.
__device__ inline uint32_t bf16_bits_rne(double x) {
  const float t = __double2float_rz(x);
  uint32_t b = __float_as_uint(t) | ((double)t != x ? 1u : 0u);
  return (b + 0x7fffu + ((b >> 16) & 1u)) >> 16;
}

// table[p][i] = (cos(p * omega_i), sin(p * omega_i)): the angle and its
// trigonometric functions are evaluated in fp64 and rounded once to fp32
// (positions reach ~1.3e5, where an fp32 angle would be off by ~1e-2 rad).
// table16 (optional) holds the same pairs rounded once from fp64 to bf16,
// packed (cos in the low half, sin in the high half) into one 32-bit word:
// the operand of the prefill's key rotation, whose products are exact in
// fp32 and whose result is rounded to bf16 anyway.
__global__ void build_table_kernel(float2* table, uint32_t* table16, int n_pos, Omega om) {
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long long)n_pos * kHalf) return;
  const int p = (int)(idx >> 6);
  const int i = (int)(idx & 63);
  double s, c;
  sincos((double)p * om.w[i], &s, &c);
  table[idx] = make_float2((float)c, (float)s);
  if (table16 != nullptr) table16[idx] = bf16_bits_rne(c) | (bf16_bits_rne(s) << 16);
}

hipError_t launch_build_table(float2* table, uint32_t* table16, int n_pos, const double* omega,
                              hipStream_t stream) {
  Omega om;
  for (int i = 0; i < kHalf; ++i) om.w[i] = omega[i];
  const long long n = (long long)n_pos * kHalf;
  const unsigned blocks = (unsigned)((n + 255) / 256);
  hipLaunchKernelGGL(build_table_kernel, dim3(blocks), dim3(256), 0, stream, table, table16, n_pos,
                     om);
  return hipGetLastError();
}

// The frequency map's tables for a packed batch (Sec. 4.5): row seq0 + p of
// sequence (seq0, L) holds (cos, sin)(p omega'_i), omega'_i = (1 - gamma_i)
// omega_i / s + gamma_i omega_i, s = max(1, L / w_pretrained), in fp32 and as
// bf16 pairs, like the base tables.  omega'_i is formed in fp64 with the
// operations, in the order, that the host uses for a single sequence, so each
// sequence's rows equal the table of a call on that sequence alone.  One
// workgroup per key-tile entry of the packed batch's plan.
struct PackedFreqArgs {
  const int4* twork;  // per key tile: (seq0, L, tile, tile0); L <= 0 marks an unused entry
  float2* table;
  uint32_t* table16;
  int w_pre;
  double omega[kHalf];
  double gamma[kHalf];
};

__global__ __launch_bounds__(256) void packed_freq_table_kernel(PackedFreqArgs a) {
#pragma clang fp contract(off)
  const int4 w = a.twork[blockIdx.x];
  if (w.y <= 0) return;
  const double s = fmax(1.0, (double)w.y / (double)a.w_pre);
  for (int idx = threadIdx.x; idx < 64 * kHalf; idx += 256) {
    const int p = w.z * 64 + (idx >> 6);
    if (p >= w.y) continue;
    const int i = idx & (kHalf - 1);
    const double om = (1.0 - a.gamma[i]) * a.omega[i] / s + a.gamma[i] * a.omega[i];
    double sn, cs;
    sincos((double)p * om, &sn, &cs);
    const size_t r = ((size_t)w.x + p) * kHalf + i;
    a.table[r] = make_float2((float)cs, (float)sn);
    a.table16[r] = bf16_bits_rne(cs) | (bf16_bits_rne(sn) << 16);
  }
}

// og: omega_i (64) then gamma_i (64), as the host computes them
hipError_t launch_packed_freq_table(const int4* twork, int nt, int w_pre, const double* og,
                                    float2* table, uint32_t* table16, hipStream_t stream) {
  PackedFreqArgs a;
  a.twork = twork;
  a.table = table;
  a.table16 = table16;
  a.w_pre = w_pre;
  for (int i = 0; i < kHalf; ++i) {
    a.omega[i] = og[i];
    a.gamma[i] = og[kHalf + i];
  }
  if (nt <= 0) return hipSuccess;
  hipLaunchKernelGGL(packed_freq_table_kernel, dim3((unsigned)nt), dim3(256), 0, stream, a);
  return hipGetLastError();
}

__global__ void debug_schedule_kernel(const int32_t* lengths, int nl, const int32_t* positions,
                                      int np, int w, int32_t* gout, int32_t* fout,
                                      int32_t* dout) {
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long long)nl * np) return;
  const int li = (int)(idx / np);
  const int pi = (int)(idx - (long long)li * np);
  const int G = group_size(lengths[li], w);
  const FastDiv gd = make_fastdiv((uint32_t)G);
  const int x = positions[pi];
  fout[idx] = remote_pos(x, gd);
  dout[idx] = pos_offset(x, gd);
  if (pi == 0) gout[li] = G;
}

hipError_t launch_debug_schedule(const int32_t* lengths, int nl, const int32_t* positions, int np,
                                 int w, int32_t* gout, int32_t* fout, int32_t* dout,
                                 hipStream_t stream) {
  const long long n = (long long)nl * np;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(debug_schedule_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                     stream, lengths, nl, positions, np, w, gout, fout, dout);
  return hipGetLastError();
}

__global__ void debug_tiles_kernel(int L, int BQ, int BK, int w0, int nqb, int nkt, int8_t* out) {
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long long)nqb * nkt) return;
  const int qb = (int)(idx / nkt);
  const int kt = (int)(idx - (long long)qb * nkt);
  const int q0 = qb * BQ, q1 = min(q0 + BQ, L) - 1;
  out[idx] = (int8_t)tile_class(visit_ranges(q0, q1, w0, BK), kt);
}

hipError_t launch_debug_tiles(int L, int BQ, int BK, int w0, int nqb, int nkt, int8_t* out,
                              hipStream_t stream) {
  const long long n = (long long)nqb * nkt;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(debug_tiles_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream,
                     L, BQ, BK, w0, nqb, nkt, out);
  return hipGetLastError();
}

}  // namespace jl
