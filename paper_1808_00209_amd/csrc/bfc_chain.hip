// A run of consecutive small binary FC layers in one launch (the classifier
// tail of Table II / Table I networks: FC layers after the last conv).
//
// Every block owns R rows of the batch and takes them through all the layers:
// its rows' packed input goes to LDS, each layer reads its input bits from
// LDS and writes its thresholded output bits back to LDS for the next layer,
// and only the last layer writes global memory (packed bits, or int32 sums
// for the logits).  No block reads another block's results, so the layers
// need no device-wide synchronisation between them.  Each block reads every
// layer's weights, which is why only layers with small weight matrices are
// chained (the caller decides).
//
// Per layer, output n is computed by T consecutive threads (T = 1 when the
// layer has at least 256 outputs, else the largest power of two with
// N * T <= 256): each XORs its share of the K words of weight row n with the
// R activation rows (LDS broadcast reads) and popcounts (Eq. 4), a
// cross-lane sum joins the T shares, and the thread holding the total applies
// the threshold and sets the output bit with an LDS OR.  A pass over the
// finished words then applies the flip bits and clears the tail.
#include "kernels.hpp"

namespace bnn {
namespace {

constexpr int kFcMaxKw = 1024;  // words of a layer input (32768 bits) held per row

struct FcChainArgs {
  FcChainLayer L[kFcChainMax];
  int32_t n;        // layers
  int32_t M;        // rows
  const uint32_t* in;
  uint32_t* out_bits;
  int32_t* out_sums;
};

template <int R, bool VEC>
__device__ __forceinline__ void fc_layer(const FcChainLayer& l, const uint32_t* act, int kw_in,
                                         uint32_t* obuf, int nw_out, int rows, int m0,
                                         bool last, const FcChainArgs& a) {
  const int tid = threadIdx.x;
  const int K = l.K, N = l.N;
  int T = 1;
  while (T < 64 && N * (2 * T) <= 256) T *= 2;
  const int per_pass = 256 / T;
  const int part = tid & (T - 1);
  const uint32_t tmask = tail_mask(K);
  const bool want_bits = !last || a.out_bits;  // thr is then non-null
  // Share of the K words for this thread: whole 4-word chunks (VEC) or words.
  const int units = VEC ? kw_in / 4 : kw_in;
  const int u0 = static_cast<int>((static_cast<int64_t>(units) * part) / T);
  const int u1 = static_cast<int>((static_cast<int64_t>(units) * (part + 1)) / T);
  for (int base = 0; base < N; base += per_pass) {
    const int n = base + tid / T;
    const bool nv = n < N;
    const uint32_t* wr = l.w + static_cast<size_t>(nv ? n : 0) * kw_in;
    const int32_t th = (nv && want_bits) ? l.thr[n] : 0;
    uint32_t cnt[R];
#pragma unroll
    for (int r = 0; r < R; ++r) cnt[r] = 0;
    if (nv) {
      for (int u = u0; u < u1; ++u) {
        if constexpr (VEC) {
          uint4 wv = *reinterpret_cast<const uint4*>(wr + 4 * u);
          if (4 * u + 3 == kw_in - 1) wv.w &= tmask;
#pragma unroll
          for (int r = 0; r < R; ++r) {
            const uint4 av = *reinterpret_cast<const uint4*>(act + r * kFcMaxKw + 4 * u);
            cnt[r] += __builtin_popcount(wv.x ^ av.x) + __builtin_popcount(wv.y ^ av.y) +
                      __builtin_popcount(wv.z ^ av.z) + __builtin_popcount(wv.w ^ av.w);
          }
        } else {
          uint32_t wv = wr[u];
          if (u == kw_in - 1) wv &= tmask;
#pragma unroll
          for (int r = 0; r < R; ++r) cnt[r] += __builtin_popcount(wv ^ act[r * kFcMaxKw + u]);
        }
      }
    }
    // Join the T shares (consecutive lanes of one wave).
#pragma unroll
    for (int r = 0; r < R; ++r)
      for (int off = 1; off < T; off <<= 1) cnt[r] += __shfl_xor(cnt[r], off);
    if (nv && part == 0) {
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if (r >= rows) break;
        const int S = K - 2 * static_cast<int>(cnt[r]);
        if (last && a.out_sums) a.out_sums[static_cast<size_t>(m0 + r) * N + n] = S;
        if (want_bits && S >= th)
          atomicOr(obuf + r * kFcMaxKw + n / 32, 1u << (31 - (n & 31)));
      }
    }
  }
  __syncthreads();
  // Flip bits and tail, then (last layer) the global store of the words.
  if (want_bits) {
    for (int i = tid; i < R * nw_out; i += 256) {
      const int r = i / nw_out, wi = i - r * nw_out;
      uint32_t wd = obuf[r * kFcMaxKw + wi];
      if (l.flip) wd ^= l.flip[wi];
      if (wi == nw_out - 1) wd &= tail_mask(N);
      if (last) {
        if (r < rows) a.out_bits[static_cast<size_t>(m0 + r) * nw_out + wi] = wd;
      } else {
        obuf[r * kFcMaxKw + wi] = wd;
      }
    }
  }
  __syncthreads();
}

template <int R, bool VEC>
__global__ __launch_bounds__(256) void bfc_chain_kernel(FcChainArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t act[2][R * kFcMaxKw];
  const int m0 = blockIdx.x * R;
  const int rows = min(R, a.M - m0);
  // The block's input rows, tail bits cleared (rows past M are zero).
  const int kw0 = (a.L[0].K + 31) >> 5;
  const uint32_t tm0 = tail_mask(a.L[0].K);
  for (int i = threadIdx.x; i < R * kw0; i += 256) {
    const int r = i / kw0, k = i - r * kw0;
    uint32_t v = r < rows ? a.in[static_cast<size_t>(m0 + r) * kw0 + k] : 0u;
    if (k == kw0 - 1) v &= tm0;
    act[0][r * kFcMaxKw + k] = v;
  }
  for (int li = 0; li < a.n; ++li) {
    const FcChainLayer& l = a.L[li];
    const int kw_in = (l.K + 31) >> 5;
    const int nw_out = (l.N + 31) >> 5;
    uint32_t* obuf = act[(li + 1) & 1];
    const bool last = li == a.n - 1;
    for (int i = threadIdx.x; i < R * nw_out; i += 256) {
      const int r = i / nw_out;
      obuf[r * kFcMaxKw + (i - r * nw_out)] = 0u;
    }
    __syncthreads();
    const uint32_t* in = act[li & 1];
    if (VEC && (kw_in & 3) == 0)
      fc_layer<R, true>(l, in, kw_in, obuf, nw_out, rows, m0, last, a);
    else
      fc_layer<R, false>(l, in, kw_in, obuf, nw_out, rows, m0, last, a);
  }
}

}  // namespace

bool bfc_chain_supported(const FcChainLayer* L, int n) {
  if (n < 1 || n > kFcChainMax) return false;
  for (int i = 0; i < n; ++i) {
    if (L[i].K < 1 || L[i].N < 1 || words_of(L[i].K) > kFcMaxKw ||
        words_of(L[i].N) > kFcMaxKw)
      return false;
    if (i + 1 < n && (L[i + 1].K != L[i].N || !L[i].thr)) return false;
  }
  return true;
}

hipError_t launch_bfc_chain(const FcChainLayer* L, int n, int64_t M, const uint32_t* in,
                            uint32_t* out_bits, int32_t* out_sums, hipStream_t s) {
  FcChainArgs a;
  for (int i = 0; i < n; ++i) a.L[i] = L[i];
  a.n = n;
  a.M = static_cast<int32_t>(M);
  a.in = in;
  a.out_bits = out_bits;
  a.out_sums = out_sums;
  // Rows per block: one block per row up to 64 rows, then up to 4 rows per
  // block (every block re-reads all the weights, so blocks are kept to ~64).
  const int R = M <= 64 ? 1 : M <= 128 ? 2 : 4;
  const dim3 grid(static_cast<unsigned>((M + R - 1) / R)), block(256);
  if (R == 1)
    bfc_chain_kernel<1, true><<<grid, block, 0, s>>>(a);
  else if (R == 2)
    bfc_chain_kernel<2, true><<<grid, block, 0, s>>>(a);
  else
    bfc_chain_kernel<4, true><<<grid, block, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace bnn
