// Verification-side helpers for a merged draft tree (Sec. 4 (iii)-(iv);
// VerifyMaskedGreedy in Algorithm 1).
//
// tree_mask: the attention mask under which one forward verifies the whole
// tree: a node attends to itself and its ancestors only.  One workgroup per
// tree; parents are staged in LDS and each thread walks one node's parent
// chain, setting bits in a register row of up to 256 bits.
//
// accept_walk: greedy acceptance given the verifier's prediction at every
// node: from the root, move to the child carrying the predicted token until
// none does; the path and the bonus token (the prediction at its last node)
// are what gets committed.  One wave per tree, the tree in LDS, each step a
// wave-wide ballot over the node slots.
//
// Both loops are bounded by max_nodes steps and ignore parent ids outside
// [0, max_nodes), so malformed trees cannot make them run away.
#include "common.hpp"
#include "internal.hpp"

namespace oil {

constexpr int kMaskWords = OIL_NODES_MAX / 32;

__global__ __launch_bounds__(256) void tree_mask_kernel(int32_t max_nodes, const int32_t* __restrict__ node_parent,
                                                        const int32_t* __restrict__ n_nodes,
                                                        uint32_t* __restrict__ mask)
{
    __shared__ int32_t par[OIL_NODES_MAX];
    const int b = blockIdx.x;
    const int words = (max_nodes + 31) / 32;
    for (int i = threadIdx.x; i < max_nodes; i += blockDim.x)
        par[i] = node_parent[(int64_t)b * max_nodes + i];
    __syncthreads();
    const int n = n_nodes[b];
    for (int i = threadIdx.x; i < max_nodes; i += blockDim.x) {
        uint32_t row[kMaskWords];
#pragma unroll
        for (int w = 0; w < kMaskWords; w++)
            row[w] = 0;
        if (i < n) {
            int j = i;
            for (int step = 0; step <= max_nodes && j >= 0 && j < max_nodes; step++) {
#pragma unroll
                for (int w = 0; w < kMaskWords; w++)
                    if (w == (j >> 5))
                        row[w] |= 1u << (j & 31);
                j = par[j];
            }
        }
        uint32_t* out = mask + ((int64_t)b * max_nodes + i) * words;
#pragma unroll
        for (int w = 0; w < kMaskWords; w++)
            if (w < words)
                out[w] = row[w];
    }
}

__global__ __launch_bounds__(64) void accept_walk_kernel(
    int32_t max_nodes, const int32_t* __restrict__ node_token, const int32_t* __restrict__ node_parent,
    const int32_t* __restrict__ n_nodes, const int32_t* __restrict__ target,
    int32_t* __restrict__ accept_len, int32_t* __restrict__ accept_nodes, int32_t* __restrict__ bonus)
{
    __shared__ int32_t tok[OIL_NODES_MAX], par[OIL_NODES_MAX], tgt[OIL_NODES_MAX];
    const int b = blockIdx.x, lane = threadIdx.x;
    const int64_t o = (int64_t)b * max_nodes;
    for (int i = lane; i < max_nodes; i += 64) {
        tok[i] = node_token[o + i];
        par[i] = node_parent[o + i];
        tgt[i] = target[o + i];
        accept_nodes[o + i] = -1;
    }
    __syncthreads();
    int n = n_nodes[b];
    n = n < max_nodes ? n : max_nodes;
    int cur = 0, len = 0;
    for (int step = 0; step < max_nodes; step++) {
        const int32_t want = tgt[cur];
        int next = -1;
        for (int base = 0; base < n; base += 64) {
            const int c = base + lane;
            const bool hit = c >= 1 && c < n && par[c] == cur && tok[c] == want;
            const uint64_t m = __ballot(hit);
            if (m) {
                next = base + __ffsll((unsigned long long)m) - 1;
                break;
            }
        }
        if (next < 0)
            break;
        if (lane == 0)
            accept_nodes[o + len] = next;
        len++;
        cur = next;
    }
    if (lane == 0) {
        accept_len[b] = len;
        bonus[b] = tgt[cur];
    }
}

hipError_t launch_tree_mask(int32_t B, int32_t max_nodes, const int32_t* node_parent,
                            const int32_t* n_nodes, uint32_t* mask, hipStream_t stream)
{
    hipLaunchKernelGGL(tree_mask_kernel, dim3(B), dim3(256), 0, stream, max_nodes, node_parent, n_nodes, mask);
    return hipGetLastError();
}

hipError_t launch_accept_walk(int32_t B, int32_t max_nodes, const int32_t* node_token,
                              const int32_t* node_parent, const int32_t* n_nodes, const int32_t* target,
                              int32_t* accept_len, int32_t* accept_nodes, int32_t* bonus,
                              hipStream_t stream)
{
    hipLaunchKernelGGL(accept_walk_kernel, dim3(B), dim3(64), 0, stream, max_nodes, node_token, node_parent,
                       n_nodes, target, accept_len, accept_nodes, bonus);
    return hipGetLastError();
}

}  // namespace oil
