// Routing-aware adaptive speculative expansion (Sec. "Routing-aware Adaptive
// Speculative Expansion"): best-first selection of draft-tree tokens by the
// utility U_i = p_i T_AR / (|E_i \ U| T_exp + C_i^draft) while U_i >= 1.
//
// One workgroup of 256 threads per tree; the whole tree state lives in LDS:
//   mask[(l*E + e) * nw + w]  bit i%32 of word w = i/32: node i predicts
//                             expert e at layer l (an inverted index: which
//                             nodes a (layer, expert) pair touches)
//   uni[l * ew + e/32]        the union U of the selected tokens' pairs
//   cnt[i]                    |E_i \ U|, kept current as U grows
//   ben[i]                    p_i, then B_i = p_i T_AR
// Phases: (1) clear, root experts into U, per-node validity; (2) one wave per
// node streams its [L][k] ids once from HBM, sets its mask bits and counts
// its distinct pairs outside U; (3) prefix confidences, resolved level by
// level; (4) the greedy loop.  Each selection costs one scan of the pair
// masks for the selected node's new pairs plus, per candidate, one mask test
// per new pair -- no per-step pass over the ids.
#include "common.h"
#include "kernels.h"

namespace s2moe {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr uint8_t kValid = 1, kAdmitted = 2;

struct Misc {
  double red_u[kWaves];
  int red_i[kWaves];
  int counter[2];
  int status;
  int pairs;
};

static_assert(sizeof(Misc) <= 128, "Misc must fit its LDS slot");

// U_i from the node's benefit, current new-pair count and C^draft, in the
// order B / (n * T_exp + c) with no fused multiply-add.
__device__ __forceinline__ double utility(double ben, int n_new, double t_exp, double c) {
#pragma clang fp contract(off)
  const double cost = (double)n_new * t_exp + c;
  return ben / cost;
}

// (u, i) beats (bu, bi): larger utility, then smaller node index.
__device__ __forceinline__ bool better(double u, int i, double bu, int bi) {
  return u > bu || (u == bu && i < bi);
}

template <int NPT>
__global__ __launch_bounds__(kThreads) void expand_kernel(ExpandArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const ExpandLds lay = expand_lds(a.N, a.L, a.E, a.k);
  double* ben = reinterpret_cast<double*>(lds + lay.ben);
  uint32_t* mask = reinterpret_cast<uint32_t*>(lds + lay.mask);
  uint32_t* uni = reinterpret_cast<uint32_t*>(lds + lay.uni);
  int* cnt = reinterpret_cast<int*>(lds + lay.cnt);
  int* list = reinterpret_cast<int*>(lds + lay.list);
  Misc* misc = reinterpret_cast<Misc*>(lds + lay.misc);
  uint8_t* state = lds + lay.state;

  const int t = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int L = a.L, E = a.E, k = a.k, N = a.N, nw = lay.nw, ew = lay.ew;
  const int Lk = L * k;
  const size_t node0 = (size_t)t * N;

  int n = a.n_nodes[t];
  int status = 0;
  if (n < 0 || n > N) {
    status |= 8;
    n = min(max(n, 0), N);
  }

  // (1) clear the masks and the union; root experts; node validity.
  const int mask_words = L * E * nw;
  for (int w = tid; w < mask_words; w += kThreads) mask[w] = 0u;
  for (int w = tid; w < L * ew; w += kThreads) uni[w] = 0u;
  if (tid == 0) {
    misc->counter[0] = 0;
    misc->counter[1] = 0;
    misc->status = 0;
    misc->pairs = 0;
  }
  int par[NPT];
  double cdr[NPT];
#pragma unroll
  for (int m = 0; m < NPT; ++m) {
    const int i = tid + m * kThreads;
    par[m] = -1;
    cdr[m] = 1.0;
    if (i < n) {
      const int pa = a.parent[node0 + i];
      const float qv = a.q[node0 + i];
      const float cv = a.c_draft[node0 + i];
      bool ok = true;
      if (!(pa == -1 || (pa >= 0 && pa < i))) { ok = false; status |= 1; }
      if (!(qv >= 0.f && qv <= 1.f)) { ok = false; status |= 2; }
      if (!(cv > 0.f && cv < INFINITY)) { ok = false; status |= 4; }
      par[m] = pa;
      cdr[m] = (double)cv;
      state[i] = ok ? kValid : 0;
      cnt[i] = 0;
      // p_i is resolved (>= 0) once its parent's is; invalid nodes are
      // resolved at once with a value nothing reads.
      ben[i] = ok ? -1.0 : 0.0;
    }
  }
  __syncthreads();
  if (status) atomicOr(&misc->status, status);
  if (a.root_eid != nullptr) {
    const int32_t* row = a.root_eid + (size_t)t * Lk;
    for (int j = tid; j < Lk; j += kThreads) {
      const int e = row[j];
      const int l = (int)(((uint32_t)j * a.k_magic) >> 20);
      if (e >= 0 && e < E) atomicOr(&uni[l * ew + (e >> 5)], 1u << (e & 31));
    }
  }
  __syncthreads();

  // (2) masks and initial counts: wave w takes nodes w, w + 4, ...; its lanes
  // stream the node's contiguous [L][k] ids.
  for (int i = wave_id(); i < n; i += kWaves) {
    const int32_t* row = a.eid + (node0 + i) * (size_t)Lk;
    const uint32_t bit = 1u << (i & 31);
    uint32_t* col = mask + (i >> 5);
    int fresh = 0;
    for (int j = lane; j < Lk; j += kWave) {
      const int e = __builtin_nontemporal_load(row + j);
      if (e >= 0 && e < E) {
        const int l = (int)(((uint32_t)j * a.k_magic) >> 20);
        const int p = l * E + e;
        const uint32_t old = atomicOr(&col[(size_t)p * nw], bit);
        if (!(old & bit) && !((uni[l * ew + (e >> 5)] >> (e & 31)) & 1u)) ++fresh;
      }
    }
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) fresh += __shfl_xor(fresh, s, kWave);
    if (lane == 0) cnt[i] = fresh;
  }

  // (3) prefix confidences, root-down: p_i = p_parent * q_i.  Each pass
  // reads resolved parents, then (after a barrier) writes, so no value is
  // read while it is being written.
  for (int pass = 0; pass <= n; ++pass) {
    double nv[NPT];
    int upd = 0;
#pragma unroll
    for (int m = 0; m < NPT; ++m) {
      const int i = tid + m * kThreads;
      nv[m] = -1.0;
      if (i < n && ben[i] < 0.0) {
        const double qi = (double)a.q[node0 + i];
        const double pp = par[m] < 0 ? 1.0 : ben[par[m]];
        if (pp >= 0.0) {
          nv[m] = pp * qi;
          upd = 1;
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int m = 0; m < NPT; ++m)
      if (nv[m] >= 0.0) ben[tid + m * kThreads] = nv[m];
    if (!__syncthreads_or(upd)) break;
  }
  double bv[NPT];
#pragma unroll
  for (int m = 0; m < NPT; ++m) {
    const int i = tid + m * kThreads;
    bv[m] = i < n ? ben[i] * a.t_ar : 0.0;
  }
  // masks, counts and ben are complete after the last pass's barrier.

  // (4) greedy selection.
  int s = 0;
  for (; s < n; ++s) {
    if (a.max_admit > 0 && s >= a.max_admit) break;
    double bu = -1.0;
    int bi = INT32_MAX;
#pragma unroll
    for (int m = 0; m < NPT; ++m) {
      const int i = tid + m * kThreads;
      if (i < n && state[i] == kValid && (par[m] < 0 || (state[par[m]] & kAdmitted))) {
        const double u = utility(bv[m], cnt[i], a.t_exp, cdr[m]);
        if (better(u, i, bu, bi)) {
          bu = u;
          bi = i;
        }
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const double ou = __shfl_xor(bu, off, kWave);
      const int oi = __shfl_xor(bi, off, kWave);
      if (better(ou, oi, bu, bi)) {
        bu = ou;
        bi = oi;
      }
    }
    if (lane == 0) {
      misc->red_u[wave_id()] = bu;
      misc->red_i[wave_id()] = bi;
    }
    __syncthreads();
    bu = misc->red_u[0];
    bi = misc->red_i[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w)
      if (better(misc->red_u[w], misc->red_i[w], bu, bi)) {
        bu = misc->red_u[w];
        bi = misc->red_i[w];
      }
    if (bi == INT32_MAX || !(bu >= 1.0)) break;  // same decision in every thread
    const int j = bi;
    int* lst = list + (s & 1) * Lk;
    int* ctr = &misc->counter[s & 1];
    if (tid == 0) {
      state[j] |= kAdmitted;
      a.order[node0 + s] = j;
      a.util[node0 + s] = bu;
      a.n_new[node0 + s] = cnt[j];
      misc->counter[(s + 1) & 1] = 0;
    }
    // New pairs of j: its mask bits at pairs not yet in U.
    const int jw = j >> 5;
    const uint32_t jb = 1u << (j & 31);
    for (int p = tid; p < L * E; p += kThreads) {
      if (mask[(size_t)p * nw + jw] & jb) {
        const int l = p / E;
        const int e = p - l * E;
        uint32_t* uw = &uni[l * ew + (e >> 5)];
        const uint32_t ub = 1u << (e & 31);
        if (!(*uw & ub)) {
          atomicOr(uw, ub);
          lst[atomicAdd(ctr, 1)] = p;
        }
      }
    }
    __syncthreads();
    // Each remaining node loses the new pairs it predicts.
    const int na = *ctr;
#pragma unroll
    for (int m = 0; m < NPT; ++m) {
      const int i = tid + m * kThreads;
      if (i < n && !(state[i] & kAdmitted)) {
        const uint32_t* col = mask + (i >> 5);
        const int sh = i & 31;
        int dec = 0;
        for (int x = 0; x < na; ++x) dec += (col[(size_t)lst[x] * nw] >> sh) & 1u;
        cnt[i] -= dec;
      }
    }
  }

  // Epilogue: padding of the per-selection outputs, union size, status.
  for (int x = s + tid; x < N; x += kThreads) {
    a.order[node0 + x] = -1;
    a.util[node0 + x] = 0.0;
    a.n_new[node0 + x] = 0;
  }
  int pc = 0;
  for (int w = tid; w < L * ew; w += kThreads) pc += __popc(uni[w]);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) pc += __shfl_xor(pc, off, kWave);
  if (lane == 0) atomicAdd(&misc->pairs, pc);
  __syncthreads();
  if (tid == 0) {
    a.n_admit[t] = s;
    a.n_pairs[t] = misc->pairs;
    a.status[t] = misc->status;
  }
}

template <int NPT>
hipError_t launch_npt(const ExpandArgs& a, size_t lds_bytes, hipStream_t s) {
  if (lds_bytes > 65536) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&expand_kernel<NPT>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             (int)lds_bytes);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(expand_kernel<NPT>, dim3(a.T), dim3(kThreads), lds_bytes, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_expand(const ExpandArgs& a, size_t lds_bytes, hipStream_t s) {
  if (a.T == 0) return hipSuccess;
  if (a.N <= kThreads) return launch_npt<1>(a, lds_bytes, s);
  if (a.N <= 2 * kThreads) return launch_npt<2>(a, lds_bytes, s);
  return launch_npt<4>(a, lds_bytes, s);
}

}  // namespace s2moe
