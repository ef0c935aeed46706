// Block-INT8 QKV records (Sec. 3.2, "Quantized communication"): the wire
// format of the sequence-parallel QKV exchange, one 400-byte record per
// (token, head).  The encoder is the sender's producer: it normalises and
// rotates q and k (Sec. 3.5, fusion group 2) and quantises q, k and v in one
// pass, so the bf16 q^, k^ never reach HBM.  The decoder writes the bf16
// tensors back (for consumers other than this library's attention, which
// decodes records in its own tile loads).  Both kernels stream: HBM-bound,
// 768 bytes read and 400 written per record (encoder), the reverse (decoder).
// The quantisation rule (scale choice, rounding) lives in sol_device.h, shared
// with the attention kernel's block-INT8 output epilogue.
#include "sol_device.h"

namespace sol {
namespace {

constexpr int kRecPerWg = 4;                 // records per workgroup
constexpr int kRecThreads = 48 * kRecPerWg;  // one thread per 16-byte chunk of q, k and v

// Eight bf16 values -> eight int8 codes of scale s (one 8-byte word).
__device__ __forceinline__ uint2 encode_chunk(uint4 y, float s) {
  float f[8];
  unpack_bf16x8(y, f);
  uint32_t w[2] = {0u, 0u};
#pragma unroll
  for (int e = 0; e < 8; ++e) w[e >> 2] |= int8_code(f[e], s) << (8 * (e & 3));
  return make_uint2(w[0], w[1]);
}

__device__ __forceinline__ float chunk_amax(uint4 y) {
  float f[8];
  unpack_bf16x8(y, f);
  float a = fabsf(f[0]);
#pragma unroll
  for (int e = 1; e < 8; ++e) a = fmaxf(a, fabsf(f[e]));
  return a;
}

// Thread t of a workgroup: record j = t / 48 of the workgroup's four, part
// p = (t / 16) % 3 (q, k, v), chunk cc = t % 16.  A part's 16 chunks sit in
// 16 aligned lanes of one wave (48 and 64 are multiples of 16), as the row
// sums of the normalisation need; a scale group is 4 aligned lanes.
// Rows are read through element strides (sb, sh, sn) shared by q, k and v,
// so a packed QKV buffer (e.g. [B][N][3][H][D]) is encoded where it lies, as
// the paper's stride-aware pack kernels do; each row's D values contiguous.
template <bool kRope>
__global__ __launch_bounds__(kRecThreads) void qkv_encode_kernel(
    const uint4* __restrict__ q, const uint4* __restrict__ k, const uint4* __restrict__ v,
    uint8_t* __restrict__ rec, int64_t n_rec, int H, SeqGrid g, const float2* __restrict__ tab,
    const float* __restrict__ q_gamma, const float* __restrict__ k_gamma, float eps,
    int64_t sb, int64_t sh, int64_t sn) {
  __shared__ uint8_t scales[kRecPerWg][12];
  const int t = threadIdx.x;
  const int j = t / 48, p = (t / 16) % 3, cc = t & 15;
  const int64_t ri = (int64_t)blockIdx.x * kRecPerWg + j;
  if (ri < n_rec) {  // uniform over the part's 16 lanes
    const int N = g.n;
    const int64_t bn = ri / H;
    const int h = (int)(ri - bn * H);
    const int64_t b = bn / N;
    const int n = (int)(bn - b * N);
    const int64_t row = b * sb + h * sh + n * sn;  // in elements, a multiple of 8
    const uint4* src = p == 0 ? q : (p == 1 ? k : v);
    const uint4 x = src[row / 8 + cc];
    uint4 y = x;
    if (p < 2) {
      const float* gamma = p == 0 ? q_gamma : k_gamma;
      const float inv = gamma ? rms_inv(row_sumsq_lanes16(chunk_sumsq(x)), eps) : 1.0f;
      Pos pos{0, 0, 0, false};
      if (kRope) pos = token_pos(n, g);
      const bool rot = kRope && pos.rot;
      y = qk_chunk(x, gamma, inv, cc, rot, tab, tab_lo_plane(tab, g), rot ? tab_pair(cc, pos, g) : 0);
    }
    float a = chunk_amax(y);
    a = fmaxf(a, __shfl_xor(a, 1));
    a = fmaxf(a, __shfl_xor(a, 2));
    const uint32_t sc = ue5m3_scale_for(a);
    uint8_t* r = rec + ri * kRecBytes;
    *reinterpret_cast<uint2*>(r + 128 * p + 8 * cc) = encode_chunk(y, ue5m3_value(sc));
    if ((cc & 3) == 0) scales[j][4 * p + (cc >> 2)] = (uint8_t)sc;
  }
  __syncthreads();
  // the record's last 16 bytes: twelve scale codes and four zero bytes
  if (t < kRecPerWg && (int64_t)blockIdx.x * kRecPerWg + t < n_rec) {
    uint32_t w[3];
#pragma unroll
    for (int i = 0; i < 3; ++i)
      w[i] = scales[t][4 * i] | scales[t][4 * i + 1] << 8 | scales[t][4 * i + 2] << 16 |
             (uint32_t)scales[t][4 * i + 3] << 24;
    uint8_t* r = rec + ((int64_t)blockIdx.x * kRecPerWg + t) * kRecBytes;
    *reinterpret_cast<uint4*>(r + kRecScales) = make_uint4(w[0], w[1], w[2], 0u);
  }
}

__global__ __launch_bounds__(kRecThreads) void qkv_decode_kernel(
    const uint8_t* __restrict__ rec, uint4* __restrict__ q, uint4* __restrict__ k,
    uint4* __restrict__ v, int64_t n_rec, int H, int N) {
  const int t = threadIdx.x;
  const int j = t / 48, p = (t / 16) % 3, cc = t & 15;
  const int64_t ri = (int64_t)blockIdx.x * kRecPerWg + j;
  if (ri >= n_rec) return;
  const int64_t bn = ri / H;
  const int h = (int)(ri - bn * H);
  const int64_t b = bn / N;
  const int n = (int)(bn - b * N);
  const size_t row = ((size_t)b * H + h) * N + n;
  uint4* dst = p == 0 ? q : (p == 1 ? k : v);
  dst[row * kChunks + cc] = rec_chunk(rec + ri * kRecBytes, p, cc);
}

}  // namespace

hipError_t launch_qkv_encode(const uint16_t* q, const uint16_t* k, const uint16_t* v, uint8_t* rec,
                             int B, int H, const SeqGrid& g, const float2* tab,
                             const float* q_gamma, const float* k_gamma, float eps,
                             int64_t sb, int64_t sh, int64_t sn, hipStream_t stream) {
  const int64_t n_rec = (int64_t)B * g.n * H;
  const dim3 grid((unsigned)((n_rec + kRecPerWg - 1) / kRecPerWg));
  const uint4* q4 = reinterpret_cast<const uint4*>(q);
  const uint4* k4 = reinterpret_cast<const uint4*>(k);
  const uint4* v4 = reinterpret_cast<const uint4*>(v);
  if (tab != nullptr)
    hipLaunchKernelGGL(qkv_encode_kernel<true>, grid, dim3(kRecThreads), 0, stream, q4, k4, v4, rec,
                       n_rec, H, g, tab, q_gamma, k_gamma, eps, sb, sh, sn);
  else
    hipLaunchKernelGGL(qkv_encode_kernel<false>, grid, dim3(kRecThreads), 0, stream, q4, k4, v4, rec,
                       n_rec, H, g, tab, q_gamma, k_gamma, eps, sb, sh, sn);
  return hipGetLastError();
}

hipError_t launch_qkv_decode(const uint8_t* rec, uint16_t* q, uint16_t* k, uint16_t* v, int B, int H,
                             int N, hipStream_t stream) {
  const int64_t n_rec = (int64_t)B * N * H;
  const dim3 grid((unsigned)((n_rec + kRecPerWg - 1) / kRecPerWg));
  hipLaunchKernelGGL(qkv_decode_kernel, grid, dim3(kRecThreads), 0, stream, rec,
                     reinterpret_cast<uint4*>(q), reinterpret_cast<uint4*>(k),
                     reinterpret_cast<uint4*>(v), n_rec, H, N);
  return hipGetLastError();
}

}  // namespace sol
