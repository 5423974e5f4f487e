// Switch-hyperedge connection count for gfx950 (Sec. 3.2 and the
// switch-hyperedge policy of Sec. 5.1; App. B.3: is_util[src, r] is 1 when
// some chunk travels from GPU src to GPU r over a switched link, and the
// uc-max / uc-min policies add gamma * sum(is_util) to the objective, gamma
// negative for uc-max and positive for uc-min).
//
// A connection is an ordered rank pair (a, b) that exchanges a chunk
// through switch vertices only. Alltoall: two ranks of a chunk's routed
// path with only switch vertices between them. Multicast: the routed paths
// of a chunk merge into its tree by first reach (destinations ascending, as
// in the evaluation kernels); a rank whose tree parent is a switch forms a
// pair with the nearest rank above it. ReduceScatter runs the trees
// backwards, so its pairs are reversed; Allreduce has both directions.
//
// One block per candidate at a time (grid-stride). The candidate's pairs
// are set in a P x P bit matrix in LDS, which is then counted.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace taccl {

namespace {

__device__ __forceinline__ void set_pair(uint32_t *bits, uint32_t a, uint32_t b, uint32_t P) {
  const uint32_t x = a * P + b;
  atomicOr(&bits[x >> 5], 1u << (x & 31));
}

template <bool kTree>
__global__ __launch_bounds__(kConnMaxThreads) void connections_kernel(ConnArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  __shared__ uint32_t total;
  const uint32_t P = (uint32_t)a.P, V = (uint32_t)a.V;
  const int C = a.C, MW = a.mask_words;
  uint32_t *bits = (uint32_t *)lds;
  // multicast: tree parent of every vertex of this thread's chunk (0xFF: not
  // reached); vertex ids are below 255
  uint8_t *par = lds + 4 * MW + threadIdx.x * V;
  for (int64_t i = blockIdx.x; i < a.n; i += gridDim.x) {
    for (int w = threadIdx.x; w < MW; w += blockDim.x) bits[w] = 0;
    if (threadIdx.x == 0) total = 0;
    __syncthreads();
    const uint8_t *rt = a.routes + (size_t)i * a.route_stride;
    for (int c = threadIdx.x; c < C; c += blockDim.x) {
      if (!kTree) {
        // chunk c = (s*P + d)*cpr + j
        const uint32_t sd = (uint32_t)c / (uint32_t)a.cpr;
        const uint32_t s = sd / P, d = sd - s * P;
        if (s == d) continue;
        const uint32_t k = rt[c];
        if (k >= a.npaths[sd]) continue;  // unrouted
        const uint32_t q = a.pair_base[sd] + k;
        uint32_t last = s;
        bool through_switch = false;
        for (uint32_t j = a.path_off[q]; j < a.path_off[q + 1]; j++) {
          const uint32_t v = a.ldst[a.path_links[j]];
          if (v >= P) {
            through_switch = true;
            continue;
          }
          if (through_switch) set_pair(bits, last, v, P);
          last = v;
          through_switch = false;
        }
      } else {
        const uint32_t o = (uint32_t)a.owner[c];
        const uint64_t pm = a.post_mask[c];
        for (uint32_t v = 0; v < V; v++) par[v] = 0xFF;
        par[o] = (uint8_t)o;
        for (uint32_t d = 0; d < P; d++) {
          if (d == o || !((pm >> d) & 1)) continue;
          const uint32_t k = rt[(size_t)c * P + d];
          const uint32_t pp = o * P + d;
          if (k >= a.npaths[pp]) continue;  // unrouted
          const uint32_t q = a.pair_base[pp] + k;
          uint32_t u = o;
          for (uint32_t j = a.path_off[q]; j < a.path_off[q + 1]; j++) {
            const uint32_t v = a.ldst[a.path_links[j]];
            if (par[v] == 0xFF) par[v] = (uint8_t)u;  // first reach
            u = v;
          }
        }
        for (uint32_t b = 0; b < P; b++) {
          if (b == o || par[b] == 0xFF) continue;
          uint32_t x = par[b];
          if (x < P) continue;
          while (x >= P) x = par[x];  // the owner is a rank, so this ends
          if (a.kind != TACCL_REDUCESCATTER) set_pair(bits, x, b, P);
          if (a.kind == TACCL_REDUCESCATTER || a.kind == TACCL_ALLREDUCE)
            set_pair(bits, b, x, P);
        }
      }
    }
    __syncthreads();
    uint32_t cnt = 0;
    for (int w = threadIdx.x; w < MW; w += blockDim.x) cnt += __popc(bits[w]);
    for (int o = 32; o > 0; o >>= 1) cnt += (uint32_t)__shfl_xor((int)cnt, o);
    if ((threadIdx.x & 63) == 0 && cnt) atomicAdd(&total, cnt);
    __syncthreads();
    if (threadIdx.x == 0) a.out[i] = total;
    __syncthreads();
  }
}

}  // namespace

int32_t connections_lds_bytes(const ConnArgs &a, int threads) {
  return 4 * a.mask_words + (a.tree ? threads * a.V : 0);
}

hipError_t launch_connections(const ConnArgs &a, int threads, int grid, hipStream_t stream) {
  if (threads < 64 || threads > kConnMaxThreads || threads % 64) return hipErrorInvalidValue;
  const void *fn = a.tree ? (const void *)connections_kernel<true>
                          : (const void *)connections_kernel<false>;
  void *args[] = {(void *)&a};
  return hipLaunchKernel(fn, dim3(grid), dim3(threads), args, connections_lds_bytes(a, threads),
                         stream);
}

}  // namespace taccl
