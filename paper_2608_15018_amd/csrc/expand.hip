// Routing-aware adaptive speculative expansion (Sec. "Routing-aware Adaptive
// Speculative Expansion"): best-first selection of draft-tree tokens by the
// utility U_i = p_i T_AR / (|E_i \ U| T_exp + C_i^draft) while U_i >= 1.
//
// One workgroup of 256 threads per tree; the tree's state lives in LDS as
// expert bitsets of EW words (E rounded up to a power of two >= 32):
//   rows[i][l][w]  the experts node i is predicted to use at layer l
//   uni[l][w]      the union U of the selected tokens' (layer, expert) pairs
//   ben[i]         p_i, then B_i = p_i T_AR;  cdr[i] = C_i^draft
//   front[]        the current candidates (parent selected or the root)
// so that repeated ids collapse by themselves, |E_i \ U| is
// sum_l popcount(rows[i][l] & ~uni[l]) and U grows by a word-wise OR.
// Phases: (1) per-node validity and the root's experts into U; (2) all
// threads stream the tree's [n][L][k] ids from HBM once (16-byte loads, many
// in flight) and set the row bits; (3) prefix confidences, resolved level by
// level; (4) the greedy loop: each step lists the candidates, each 16-lane
// row of each wave scores one candidate at a time (a lane per layer), the
// block takes the largest U_i (ties: smaller index) and, if U_i >= 1, ORs
// the node's rows into U.
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
  int red_n[kWaves];
  int counter[2];
  int any[2];
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

__device__ __forceinline__ int wave_sum_int(int v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}

// Sum over each 16-lane row (DPP row shifts); the total lands in the row's
// last lane.
__device__ __forceinline__ int row16_sum(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);  // row_shr:8
  return v;
}

__device__ __forceinline__ double readlane_f64(double v, int lane) {
  const uint64_t u = __double_as_longlong(v);
  const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)u, lane);
  const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), lane);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// popcount(a & ~b) over one EW-word bitset pair, read as aligned vectors.
template <int EW>
__device__ __forceinline__ int count_new(const uint32_t* a, const uint32_t* b) {
  int c = 0;
  if constexpr (EW == 1) {
    c = __popc(a[0] & ~b[0]);
  } else if constexpr (EW == 2) {
    const uint64_t x = *reinterpret_cast<const uint64_t*>(a);
    const uint64_t y = *reinterpret_cast<const uint64_t*>(b);
    c = __popcll(x & ~y);
  } else {
#pragma unroll
    for (int q = 0; q < EW / 4; ++q) {
      const u32x4 x = reinterpret_cast<const u32x4*>(a)[q];
      const u32x4 y = reinterpret_cast<const u32x4*>(b)[q];
#pragma unroll
      for (int w = 0; w < 4; ++w) c += __popc(x[w] & ~y[w]);
    }
  }
  return c;
}

// Where tree t's ids lie: n * L * k int32 from element e0 of eid (n = the
// tree's node count, clamped to [0, N]); the first `head` ids precede the
// first 16-byte boundary, then `nch` whole 16-byte chunks, then the rest.
struct IdRun {
  int n, bad_count, total, head, nch;
  size_t e0;
};

__device__ __forceinline__ IdRun id_run(const ExpandArgs& a, int t) {
  IdRun r;
  const int n = a.n_nodes[t];
  r.bad_count = n < 0 || n > a.N;
  r.n = min(max(n, 0), a.N);
  r.e0 = (size_t)t * a.N * (size_t)(a.L * a.k);
  r.total = r.n * a.L * a.k;
  // eid is 16-byte aligned, so the run's first 16-byte boundary is at
  // element (4 - e0 mod 4) mod 4.
  r.head = min(r.total, (int)((4u - (uint32_t)(r.e0 & 3u)) & 3u));
  r.nch = (r.total - r.head) >> 2;
  return r;
}

// Chunks c = tid + 256 u (u < PF) of a tree's run, loaded ahead.
template <int PF>
__device__ __forceinline__ void prefetch_ids(const ExpandArgs& a, const IdRun& r, u32x4 (&pf)[PF]) {
  const u32x4* body = reinterpret_cast<const u32x4*>(a.eid + r.e0 + r.head);
#pragma unroll
  for (int u = 0; u < PF; ++u) {
    const int c = (int)threadIdx.x + u * kThreads;
    if (c < r.nch) pf[u] = __builtin_nontemporal_load(body + c);
  }
}

// A persistent workgroup takes trees blockIdx.x, + gridDim.x, ...  With
// PF > 0, while it runs one tree's greedy loop the first PF * 256 chunks of
// its next tree's ids are already on their way into registers (used when a
// tree's LDS leaves room for one workgroup per CU anyway; smaller trees run
// several workgroups per CU instead).
template <int NPT, int EW, int PF>
__global__ __launch_bounds__(kThreads) void expand_kernel(ExpandArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const ExpandLds lay = expand_lds(a.N, a.L, a.E, a.k);
  double* ben = reinterpret_cast<double*>(lds + lay.ben);
  uint32_t* rows = reinterpret_cast<uint32_t*>(lds + lay.rows);
  uint32_t* uni = reinterpret_cast<uint32_t*>(lds + lay.uni);
  float* cdr = reinterpret_cast<float*>(lds + lay.cdr);
  int* front = reinterpret_cast<int*>(lds + lay.front);
  Misc* misc = reinterpret_cast<Misc*>(lds + lay.misc);
  uint8_t* state = lds + lay.state;

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int L = a.L, E = a.E, k = a.k, N = a.N;
  const int Lk = L * k;

  u32x4 pf[PF > 0 ? PF : 1];
  if constexpr (PF > 0)
    if ((int)blockIdx.x < a.T) prefetch_ids<PF>(a, id_run(a, blockIdx.x), pf);

  // Without prefetch the grid has one workgroup per tree: one pass.
  const int t_step = PF > 0 ? (int)gridDim.x : a.T;
  for (int t = blockIdx.x; t < a.T; t += t_step) {
  const size_t node0 = (size_t)t * N;
  const IdRun run = id_run(a, t);
  const int n = run.n;
  int status = run.bad_count ? 8 : 0;

  // (1) per-node records and the root's ids: one round of loads.
  int par[NPT];
  double qd[NPT];
#pragma unroll
  for (int m = 0; m < NPT; ++m) {
    const int i = tid + m * kThreads;
    par[m] = -1;
    qd[m] = 0.0;
    if (i < n) {
      const int pa = a.parent[node0 + i];
      const float qv = a.q[node0 + i];
      const float cv = a.c_draft[node0 + i];
      bool ok = true;
      if (!(pa == -1 || (pa >= 0 && pa < i))) { ok = false; status |= 1; }
      if (!(qv >= 0.f && qv <= 1.f)) { ok = false; status |= 2; }
      if (!(cv > 0.f && cv < INFINITY)) { ok = false; status |= 4; }
      par[m] = pa;
      qd[m] = (double)qv;
      state[i] = ok ? kValid : 0;
      cdr[i] = cv;
      // p_i is resolved (>= 0) once its parent's is; invalid nodes are
      // resolved at once with a value nothing reads.
      ben[i] = ok ? -1.0 : 0.0;
    }
  }
  constexpr int kRootPer = 4096 / kThreads;  // L * k <= 4096
  int rv[kRootPer];
#pragma unroll
  for (int r = 0; r < kRootPer; ++r) {
    const int j = tid + r * kThreads;
    rv[r] = -1;
    if (a.root_eid != nullptr && j < Lk) rv[r] = a.root_eid[(size_t)t * Lk + j];
  }
  // Clear the n nodes' row bitsets (16-byte aligned, EW-word rows) and the
  // union.
  {
    const int words = n * L * EW;
    u32x4* r4 = reinterpret_cast<u32x4*>(rows);
    for (int w = tid; w < (words >> 2); w += kThreads) r4[w] = u32x4{0u, 0u, 0u, 0u};
    for (int w = (words & ~3) + tid; w < words; w += kThreads) rows[w] = 0u;
    for (int w = tid; w < L * EW; w += kThreads) uni[w] = 0u;
  }
  if (tid == 0) {
    misc->counter[0] = 0;
    misc->counter[1] = 0;
    misc->any[0] = 0;
    misc->status = 0;
    misc->pairs = 0;
  }
  __syncthreads();
  if (status) atomicOr(&misc->status, status);
#pragma unroll
  for (int r = 0; r < kRootPer; ++r) {
    const int j = tid + r * kThreads;
    const int e = rv[r];
    if (j < Lk && e >= 0 && e < E) {
      const int l = (int)(((uint64_t)j * a.k_div) >> 42);
      atomicOr(&uni[l * EW + (e >> 5)], 1u << (e & 31));
    }
  }

  // (2) the tree's ids, one contiguous node-major run of n * L * k int32:
  // id f belongs to row f / k (= node * L + layer); ids outside [0, E) are
  // padding.
  const int32_t* src = a.eid + run.e0;
  // Sets bit e of the row's bitset; padding ORs 0 into word 0 (no branch).
  auto set_bit = [&](uint32_t row, int e) {
    const bool ok = (uint32_t)e < (uint32_t)E;
    const uint32_t w = ok ? row * EW + ((uint32_t)e >> 5) : 0u;
    atomicOr(&rows[w], ok ? 1u << (e & 31) : 0u);
  };
  auto row_of = [&](uint32_t f) { return (uint32_t)(((uint64_t)f * a.k_div) >> 42); };
  const int head = run.head, nch = run.nch;
  for (int f = tid; f < head; f += kThreads) set_bit(row_of(f), src[f]);
  const u32x4* body = reinterpret_cast<const u32x4*>(src + head);
  // With head == 0 and k a multiple of 4, the four ids of a chunk share a row.
  const bool same_row = head == 0 && (k & 3) == 0;
  auto place_chunk = [&](int c, const u32x4& v) {
    const uint32_t f = head + 4 * c;
    uint32_t row = row_of(f);
    if (same_row) {
#pragma unroll
      for (int x = 0; x < 4; ++x) set_bit(row, (int)v[x]);
    } else {
      uint32_t pos = f - row * k;  // position of the first id in its row
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        set_bit(row, (int)v[x]);
        if (++pos == (uint32_t)k) {
          pos = 0;
          ++row;
        }
      }
    }
  };
  // The prefetched chunks, then the rest of the run in batches.
  if constexpr (PF > 0) {
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      const int c = tid + u * kThreads;
      if (c < nch) place_chunk(c, pf[u]);
    }
  }
  constexpr int kBatch = 16;
  for (int c0 = PF * kThreads; c0 < nch; c0 += kThreads * kBatch) {
    u32x4 v[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int c = c0 + tid + u * kThreads;
      if (c < nch) v[u] = __builtin_nontemporal_load(body + c);
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int c = c0 + tid + u * kThreads;
      if (c < nch) place_chunk(c, v[u]);
    }
  }
  for (int f = head + 4 * nch + tid; f < run.total; f += kThreads) set_bit(row_of(f), src[f]);
  // This tree's ids are placed: start loading the next tree's.
  if constexpr (PF > 0)
    if (t + t_step < a.T) prefetch_ids<PF>(a, id_run(a, t + t_step), pf);

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
        const double pp = par[m] < 0 ? 1.0 : ben[par[m]];
        if (pp >= 0.0) {
          nv[m] = pp * qd[m];
          upd = 1;
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int m = 0; m < NPT; ++m)
      if (nv[m] >= 0.0) ben[tid + m * kThreads] = nv[m];
    // "any node resolved in this pass", double-buffered across passes
    if (upd) misc->any[pass & 1] = 1;
    if (tid == 0) misc->any[(pass + 1) & 1] = 0;
    __syncthreads();
    if (!misc->any[pass & 1]) break;
  }
  // B_i = p_i T_AR (each thread its own nodes; read by others after the
  // first barrier of the loop).
#pragma unroll
  for (int m = 0; m < NPT; ++m) {
    const int i = tid + m * kThreads;
    if (i < n) ben[i] = ben[i] * a.t_ar;
  }

  // (4) greedy selection.
  const int sub = lane & 15;
  int s = 0;
  for (; s < n; ++s) {
    if (a.max_admit > 0 && s >= a.max_admit) break;
    // Candidates: valid, unselected, parent selected or the root.
    int* ctr = &misc->counter[s & 1];
#pragma unroll
    for (int m = 0; m < NPT; ++m) {
      const int i = tid + m * kThreads;
      if (i < n && state[i] == kValid && (par[m] < 0 || (state[par[m]] & kAdmitted)))
        front[atomicAdd(ctr, 1)] = i;
    }
    __syncthreads();
    const int nf = *ctr;
    if (tid == 0) misc->counter[(s + 1) & 1] = 0;
    // Each 16-lane row of each wave scores one candidate at a time; the
    // row's last lane keeps the row's best.
    double bu = -1.0;
    int bi = INT32_MAX, bn = 0;
    for (int x0 = wave_id() * 4; x0 < nf; x0 += kWaves * 4) {
      const int x = x0 + (lane >> 4);
      int c = 0, i = 0;
      if (x < nf) {
        i = front[x];
        const uint32_t* ri = rows + (size_t)i * L * EW;
        for (int l = sub; l < L; l += 16) c += count_new<EW>(ri + l * EW, uni + l * EW);
      }
      c = row16_sum(c);
      if (x < nf && sub == 15) {
        const double u = utility(ben[i], c, a.t_exp, (double)cdr[i]);
        if (better(u, i, bu, bi)) {
          bu = u;
          bi = i;
          bn = c;
        }
      }
    }
    // The wave's best of its four row leaders.
    {
      double wu = readlane_f64(bu, 15);
      int wi = __builtin_amdgcn_readlane(bi, 15), wn = __builtin_amdgcn_readlane(bn, 15);
#pragma unroll
      for (int g = 1; g < 4; ++g) {
        const double gu = readlane_f64(bu, 16 * g + 15);
        const int gi = __builtin_amdgcn_readlane(bi, 16 * g + 15);
        if (better(gu, gi, wu, wi)) {
          wu = gu;
          wi = gi;
          wn = __builtin_amdgcn_readlane(bn, 16 * g + 15);
        }
      }
      bu = wu;
      bi = wi;
      bn = wn;
    }
    if (lane == 0) {
      misc->red_u[wave_id()] = bu;
      misc->red_i[wave_id()] = bi;
      misc->red_n[wave_id()] = bn;
    }
    __syncthreads();
    bu = misc->red_u[0];
    bi = misc->red_i[0];
    bn = misc->red_n[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w)
      if (better(misc->red_u[w], misc->red_i[w], bu, bi)) {
        bu = misc->red_u[w];
        bi = misc->red_i[w];
        bn = misc->red_n[w];
      }
    if (bi == INT32_MAX || !(bu >= 1.0)) break;  // same decision in every thread
    const int j = bi;
    if (tid == 0) {
      state[j] |= kAdmitted;
      a.order[node0 + s] = j;
      a.util[node0 + s] = bu;
      a.n_new[node0 + s] = bn;
    }
    // U gains the selected node's rows (one word per thread).
    const uint32_t* rj = rows + (size_t)j * L * EW;
    for (int w = tid; w < L * EW; w += kThreads) uni[w] |= rj[w];
    __syncthreads();
  }

  // Epilogue: padding of the per-selection outputs, union size, status.
  for (int x = s + tid; x < N; x += kThreads) {
    a.order[node0 + x] = -1;
    a.util[node0 + x] = 0.0;
    a.n_new[node0 + x] = 0;
  }
  int pc = 0;
  for (int w = tid; w < L * EW; w += kThreads) pc += __popc(uni[w]);
  pc = wave_sum_int(pc);
  if (lane == 0) atomicAdd(&misc->pairs, pc);
  __syncthreads();
  if (tid == 0) {
    a.n_admit[t] = s;
    a.n_pairs[t] = misc->pairs;
    a.status[t] = misc->status;
  }
  }  // trees
}

template <int NPT, int EW, int PF>
hipError_t launch_pf(const ExpandArgs& a, size_t lds_bytes, hipStream_t s) {
  const void* fn = reinterpret_cast<const void*>(&expand_kernel<NPT, EW, PF>);
  if (lds_bytes > 65536) {
    const hipError_t e =
        hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes);
    if (e != hipSuccess) return e;
  }
  // With prefetch, one persistent workgroup per resident slot (at most one
  // per tree); without, one workgroup per tree.
  int grid = a.T;
  if (PF > 0) {
    int per_cu = 0, dev = 0, cus = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kThreads, lds_bytes);
    if (e == hipSuccess) e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    grid = max(1, min(a.T, max(1, per_cu) * cus));
  }
  hipLaunchKernelGGL((expand_kernel<NPT, EW, PF>), dim3(grid), dim3(kThreads), lds_bytes, s, a);
  return hipGetLastError();
}

// Prefetch only when a tree's LDS already limits a CU to one workgroup.
constexpr size_t kLdsPerCu = 160 * 1024;

template <int NPT, int EW>
hipError_t launch_ew(const ExpandArgs& a, size_t lds_bytes, hipStream_t s) {
  return 2 * lds_bytes > kLdsPerCu ? launch_pf<NPT, EW, 32>(a, lds_bytes, s)
                                   : launch_pf<NPT, EW, 0>(a, lds_bytes, s);
}

template <int NPT>
hipError_t launch_npt(const ExpandArgs& a, size_t lds_bytes, hipStream_t s) {
  switch (expand_words(a.E)) {
    case 1: return launch_ew<NPT, 1>(a, lds_bytes, s);
    case 2: return launch_ew<NPT, 2>(a, lds_bytes, s);
    case 4: return launch_ew<NPT, 4>(a, lds_bytes, s);
    case 8: return launch_ew<NPT, 8>(a, lds_bytes, s);
    case 16: return launch_ew<NPT, 16>(a, lds_bytes, s);
    case 32: return launch_ew<NPT, 32>(a, lds_bytes, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_expand(const ExpandArgs& a, size_t lds_bytes, hipStream_t s) {
  if (a.T == 0) return hipSuccess;
  if (a.N <= kThreads) return launch_npt<1>(a, lds_bytes, s);
  if (a.N <= 2 * kThreads) return launch_npt<2>(a, lds_bytes, s);
  return launch_npt<4>(a, lds_bytes, s);
}

}  // namespace s2moe
