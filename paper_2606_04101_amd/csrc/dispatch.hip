// Step 3 — token-to-replica assignment and dispatch permutation of one
// source rank (Sec. 5.2 Token Assignment), then the bf16 row scatter.
//
// Layout (two launches, integer only):
//   k_dl_hist  : workgroup c < n_chunks counts the expert ids of slots
//                [c*2048, (c+1)*2048); the last workgroup turns row `rank` of
//                the reroute split into block sizes (t, p), their exclusive
//                prefix block_off, and per CSR entry the cumulative quota C
//                and the first row minus the entry's starting ordinal.
//   k_dl_rows  : workgroup c sums the histograms of chunks < c (its base
//                ordinal per expert), then each wave ranks its 128 slots
//                stably with ballot matches (wave-private running counts in
//                LDS, scanned across waves), finds the first instance whose
//                cumulative quota exceeds the ordinal and writes the row.
// Scatter (bandwidth bound): persistent waves walk the tokens; a wave holds
//   one token's row in registers (16-byte non-temporal loads) while the next
//   token's row is being loaded, and stores each 1 KiB chunk to all k
//   destination rows before the next chunk, with sc1 buffer stores.  The
//   rows are a permutation of the send buffer, and writing such a
//   permutation of 14 KiB rows measures about 5.2 TB/s on its own, against
//   6.5 TB/s for a sequential stream; rows past the routed count are
//   zero-filled.
#include "common.hpp"
#include "kernels.hpp"

namespace uep {

constexpr int kDlThreads = 1024;
constexpr int kDlWaves = kDlThreads / kWave;
constexpr int kSlotsPerWave = kDispatchChunk / kDlWaves;  // 128
constexpr int kMaxBlocks = 2048;                           // R * S

static_assert(kSlotsPerWave % kWave == 0, "chunk must split into wave steps");
// CSR columns (E + R * n_slot <= 1024 + 256) and start pointers (E + 1) per
// thread when a 1024-thread workgroup stages them
constexpr int kLutIters = 2;
constexpr int kSumBatch = 16;  // chunk histograms summed per batch of loads
static_assert(kLutIters * kDlThreads >= 1024 + 256 && kLutIters * kDlThreads >= 1024 + 1,
              "the lookup tables fit the staging loops");
constexpr int kSteps = kSlotsPerWave / kWave;  // 64-slot steps per wave

size_t dispatch_ws_bytes(int64_t V, int32_t E, int32_t ncol) {
  const int64_t n_chunks = (V + kDispatchChunk - 1) / kDispatchChunk;
  const int64_t ints = n_chunks * E + 2 * static_cast<int64_t>(ncol) + E;
  return static_cast<size_t>((ints * 4 + 255) / 256 * 256);
}

DispatchWs dispatch_ws(void *ws, int64_t V, int32_t E, int32_t ncol) {
  DispatchWs w;
  w.n_chunks = (V + kDispatchChunk - 1) / kDispatchChunk;
  int32_t *p = static_cast<int32_t *>(ws);
  w.hist = p;
  p += w.n_chunks * E;
  w.ent_cum = p;
  p += ncol;
  w.ent_base = p;
  p += ncol;
  w.exp_tot = p;
  return w;
}

struct DlArgs {
  const int32_t *topk;
  int64_t V;
  int32_t rank, R, E, NS, nm, S, ncol, nbits;
  int32_t stage_lut;  // copy host_ptr / entry tables into LDS
  const int32_t *hp, *hr, *hs, *q;  // q = reroute row of `rank`
  int32_t *row_of_slot;
  int64_t *block_off;
  DispatchWs ws;
  int32_t *status;
};

__global__ void __launch_bounds__(kDlThreads) k_dl_hist(DlArgs a) {
  extern __shared__ int32_t lds[];
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const int E = a.E;
  if (blockIdx.x < a.ws.n_chunks) {
    int32_t *hist = lds;  // [kDlWaves][E]
    for (int i = tid; i < kDlWaves * E; i += kDlThreads) hist[i] = 0;
    __syncthreads();
    const int64_t c0 = static_cast<int64_t>(blockIdx.x) * kDispatchChunk;
    int32_t *wh = hist + wave * E;
    bool bad = false;
    int32_t ev[kSteps];
#pragma unroll
    for (int s = 0; s < kSteps; ++s) {
      const int64_t i = c0 + wave * kSlotsPerWave + s * kWave + lane;
      ev[s] = i < a.V ? a.topk[i] : -1;
    }
#pragma unroll
    for (int s = 0; s < kSteps; ++s) {
      const int32_t e = ev[s];
      if (e >= 0 && e < E) atomicAdd(wh + e, 1);
      bad |= e < -1 || e >= E;
    }
    if (bad) report(a.status, ULTRAEP_EDATA);
    __syncthreads();
    int32_t *dst = a.ws.hist + blockIdx.x * static_cast<int64_t>(E);
    for (int e = tid; e < E; e += kDlThreads) {
      int s = 0;
      for (int w = 0; w < kDlWaves; ++w) s += hist[w * E + e];
      dst[e] = s;
    }
    return;
  }
  // ---- layout workgroup: block sizes, offsets, entry lookup tables ----
  // Every input is requested at once (indices clamped into range, no branch
  // between the loads) and staged in LDS: the CSR start pointers and, per
  // CSR column, the host rank, its slot and this rank's share.
  const int ncol = a.ncol;
  int32_t *cnt = lds;                  // [R*S]
  int32_t *tmp = lds + kMaxBlocks;     // [kDlWaves]
  int32_t *l_hp = tmp + kDlWaves + 1;  // [E + 1]
  int32_t *l_hr = l_hp + E + 1;        // [ncol]
  int32_t *l_hs = l_hr + ncol;         // [ncol]
  int32_t *l_q = l_hs + ncol;          // [ncol]
  int vhp[kLutIters], vhr[kLutIters], vhs[kLutIters], vq[kLutIters];
#pragma unroll
  for (int u = 0; u < kLutIters; ++u) {
    if (u * kDlThreads <= E) vhp[u] = a.hp[min(u * kDlThreads + tid, E)];
    if (u * kDlThreads < ncol) {
      const int j = min(u * kDlThreads + tid, ncol - 1);
      vhr[u] = a.hr[j];
      vhs[u] = a.hs[j];
      vq[u] = a.q[j];
    }
  }
  const int nblk = a.R * a.S;
  for (int b = tid; b < nblk; b += kDlThreads) cnt[b] = 0;
#pragma unroll
  for (int u = 0; u < kLutIters; ++u) {
    const int i = u * kDlThreads + tid;
    if (i <= E) l_hp[i] = vhp[u];
    if (i < ncol) {
      l_hr[i] = vhr[u];
      l_hs[i] = vhs[u];
      l_q[i] = vq[u];
    }
  }
  __syncthreads();
  // the CSR must start at 0, never decrease and end within the columns,
  // so every entry index below is inside the tables
  const int total = l_hp[E];
  bool bad = l_hp[0] != 0 || total < E || total > ncol;
  for (int e = tid; e < E; e += kDlThreads) bad |= l_hp[e] > l_hp[e + 1];
  if (__syncthreads_or(bad)) {  // not a plan of this group
    if (tid == 0) report(a.status, ULTRAEP_EDATA);
    return;
  }
  for (int j = tid; j < total; j += kDlThreads) {
    const int t = l_hr[j], p = l_hs[j];
    if (t >= 0 && t < a.R && p >= 0 && p < a.S) cnt[t * a.S + p] = l_q[j];
    else report(a.status, ULTRAEP_EDATA);
  }
  __syncthreads();
  // exclusive scan of cnt (two elements per thread) into int64 offsets
  const int b0 = 2 * tid, b1 = 2 * tid + 1;
  const int v0 = b0 < nblk ? cnt[b0] : 0, v1 = b1 < nblk ? cnt[b1] : 0;
  const int incl = wave_scan_incl(v0 + v1);
  if (lane == kWave - 1) tmp[wave] = incl;
  __syncthreads();
  if (tid == 0) {
    int run = 0;
    for (int w = 0; w < kDlWaves; ++w) {
      int t = tmp[w];
      tmp[w] = run;
      run += t;
    }
  }
  __syncthreads();
  const int ex0 = tmp[wave] + incl - v0 - v1;
  __syncthreads();
  // reuse cnt as offsets
  if (b0 < nblk) cnt[b0] = ex0;
  if (b1 < nblk) cnt[b1] = ex0 + v0;
  if (b0 < nblk) a.block_off[b0] = ex0;
  if (b1 < nblk) a.block_off[b1] = ex0 + v0;
  if (b1 == nblk || b0 == nblk) a.block_off[nblk] = ex0 + (b0 == nblk ? 0 : v0);
  __syncthreads();
  for (int e = tid; e < E; e += kDlThreads) {
    int C = 0;
    for (int j = l_hp[e]; j < l_hp[e + 1]; ++j) {
      const int t = l_hr[j], p = l_hs[j];
      const bool ok = t >= 0 && t < a.R && p >= 0 && p < a.S;
      a.ws.ent_base[j] = (ok ? cnt[t * a.S + p] : 0) - C;
      C += l_q[j];
      a.ws.ent_cum[j] = C;
    }
    a.ws.exp_tot[e] = C;
  }
}

__global__ void __launch_bounds__(kDlThreads) k_dl_rows(DlArgs a) {
  extern __shared__ int32_t lds[];
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const int E = a.E, ncol = a.ncol;
  const int c = blockIdx.x;
  int32_t *whist = lds;  // [kDlWaves][E]
  int32_t *base = lds + kDlWaves * E;
  // Every input is requested at once (indices clamped into range, no branch
  // between the loads), so the workgroup waits for memory once: its slots'
  // expert ids, the histograms of the chunks before it (of every chunk in
  // workgroup 0, which checks them against the expected totals) and the
  // instance lookup tables.
  const int64_t s0 = static_cast<int64_t>(c) * kDispatchChunk + wave * kSlotsPerWave;
  int32_t ev[kSteps];
#pragma unroll
  for (int s = 0; s < kSteps; ++s) ev[s] = a.topk[min(s0 + s * kWave + lane, a.V - 1)];
  const int e_t = min(tid, E - 1);  // this thread's expert for the sums (tid < E)
  const int nsum = c == 0 ? static_cast<int>(a.ws.n_chunks) : c;
  const int32_t *h = a.ws.hist + e_t;
  int hv[kSumBatch];
#pragma unroll
  for (int u = 0; u < kSumBatch; ++u) hv[u] = h[min(u, nsum - 1) * static_cast<int64_t>(E)];
  const int exp_tot = c == 0 ? a.ws.exp_tot[e_t] : 0;
  int vhp[kLutIters], vcum[kLutIters], vbase[kLutIters];
  if (a.stage_lut) {
#pragma unroll
    for (int u = 0; u < kLutIters; ++u) {
      if (u * kDlThreads <= E) vhp[u] = a.hp[min(u * kDlThreads + tid, E)];
      if (u * kDlThreads < ncol) {
        const int jj = min(u * kDlThreads + tid, ncol - 1);
        vcum[u] = a.ws.ent_cum[jj];
        vbase[u] = a.ws.ent_base[jj];
      }
    }
  }
#pragma unroll
  for (int s = 0; s < kSteps; ++s)
    if (s0 + s * kWave + lane >= a.V) ev[s] = -1;
  // instance lookup tables, staged in LDS when they fit
  const int32_t *l_hp = a.hp, *l_cum = a.ws.ent_cum, *l_base = a.ws.ent_base;
  if (a.stage_lut) {
    int32_t *p = base + E;
#pragma unroll
    for (int u = 0; u < kLutIters; ++u) {
      const int ii = u * kDlThreads + tid;
      if (ii <= E) p[ii] = vhp[u];
      if (ii < ncol) {
        p[E + 1 + ii] = vcum[u];
        p[E + 1 + ncol + ii] = vbase[u];
      }
    }
    l_hp = p;
    l_cum = p + E + 1;
    l_base = p + E + 1 + ncol;
  }
  // base ordinals: sums over the earlier chunks' histograms (further batches
  // of kSumBatch loads when there are more chunks than one batch)
  if (tid < E) {
    int s = 0, tot = 0;
#pragma unroll
    for (int u = 0; u < kSumBatch; ++u) {
      const int v = u < nsum ? hv[u] : 0;
      s += u < c ? v : 0;
      tot += v;
    }
    for (int c0 = kSumBatch; c0 < nsum; c0 += kSumBatch) {
      int w[kSumBatch];
#pragma unroll
      for (int u = 0; u < kSumBatch; ++u) w[u] = h[min(c0 + u, nsum - 1) * static_cast<int64_t>(E)];
#pragma unroll
      for (int u = 0; u < kSumBatch; ++u) {
        const int v = c0 + u < nsum ? w[u] : 0;
        s += c0 + u < c ? v : 0;
        tot += v;
      }
    }
    base[tid] = s;
    if (c == 0 && tot != exp_tot) report(a.status, ULTRAEP_EDATA);
  }
  for (int i = tid; i < kDlWaves * E; i += kDlThreads) whist[i] = 0;
  __syncthreads();
  int32_t *wh = whist + wave * E;
  // pass 1: per-wave counts
#pragma unroll
  for (int s = 0; s < kSteps; ++s) {
    const int32_t e = ev[s];
    if (e >= 0 && e < E) atomicAdd(wh + e, 1);
  }
  __syncthreads();
  for (int e = tid; e < E; e += kDlThreads) {
    int run = base[e];
    for (int w = 0; w < kDlWaves; ++w) {
      int t = whist[w * E + e];
      whist[w * E + e] = run;
      run += t;
    }
  }
  __syncthreads();
  // pass 2: stable ordinals, instance lookup, rows
  for (int s = 0; s < kSteps; ++s) {
    const int64_t i = s0 + s * kWave + lane;
    const int32_t e = ev[s];
    const bool valid = e >= 0 && e < E;
    const uint64_t act = ballot(valid);
    if (act == 0) {
      if (i < a.V) a.row_of_slot[i] = -1;
      continue;
    }
    const uint64_t m = match_any(static_cast<uint32_t>(valid ? e : 0), a.nbits, act);
    int row = -1;
    if (valid) {
      const int below = popc_below(m);
      const int ord = wh[e] + below;
      if (below == 0) wh[e] += __popcll(m);
      // entry range of e, clamped to the tables (a CSR that is not a plan
      // of this group cannot send the search outside them)
      const int j1 = min(max(l_hp[e + 1], 0), a.ncol);
      int j = min(max(l_hp[e], 0), j1);
      while (j < j1 && l_cum[j] <= ord) ++j;
      if (j < j1) row = l_base[j] + ord;
      // a plan row that does not match these ids can point past the buffer
      if (row < 0 || row >= a.V) {
        row = -1;
        report(a.status, ULTRAEP_EDATA);
      }
    }
    if (i < a.V) a.row_of_slot[i] = row;
  }
}

hipError_t launch_dispatch_layout(const int32_t *topk, int64_t V, int32_t rank,
                                  const ultraep_group &g,
                                  const ultraep_plan_buf &plan,
                                  int32_t *row_of_slot, int64_t *block_off,
                                  const DispatchWs &ws, int32_t *status,
                                  hipStream_t stream) {
  DlArgs a;
  a.topk = topk;
  a.V = V;
  a.rank = rank;
  a.R = g.R;
  a.E = g.E;
  a.NS = g.n_slot;
  a.nm = g.E / g.R;
  a.S = a.nm + g.n_slot;
  a.ncol = g.E + g.R * g.n_slot;
  a.nbits = bits_for(g.E);
  a.hp = plan.host_ptr;
  a.hr = plan.host_rank;
  a.hs = plan.host_pslot;
  a.q = plan.reroute + static_cast<int64_t>(rank) * a.ncol;
  a.row_of_slot = row_of_slot;
  a.block_off = block_off;
  a.ws = ws;
  a.status = status;
  a.stage_lut = 0;
  const size_t lds_hist = sizeof(int32_t) * kDlWaves * g.E;
  const size_t lds_lay =
      sizeof(int32_t) * (kMaxBlocks + kDlWaves + 1 + g.E + 1 + 3 * static_cast<size_t>(a.ncol));
  hipLaunchKernelGGL(k_dl_hist, dim3(ws.n_chunks + 1), dim3(kDlThreads),
                     lds_hist > lds_lay ? lds_hist : lds_lay, stream, a);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || ws.n_chunks == 0) return err;
  size_t lds_rows = sizeof(int32_t) * (kDlWaves + 1) * g.E;
  const size_t lut = sizeof(int32_t) * (g.E + 1 + 2 * static_cast<size_t>(a.ncol));
  if (lds_rows + lut <= 64 * 1024) {
    lds_rows += lut;
    a.stage_lut = 1;
  }
  hipLaunchKernelGGL(k_dl_rows, dim3(ws.n_chunks), dim3(kDlThreads), lds_rows, stream, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------- scatter

constexpr int kScThreads = 256;
constexpr int kScWaves = kScThreads / kWave;
// Resident workgroups of the streaming scatter (two per CU); each wave then
// walks tokens t, t + 2048, ...  Measured against one wave per token and
// against 256 to 1024 workgroups on the DeepSeek-V3-shaped layer.
constexpr int kScGrid = 512;
// dword 3 of a raw buffer resource (32-bit data format) and the store cache
// policy: sc1 streams the rows out at the device scope.  Buffer stores with
// sc1 measured 3-4 % faster than plain or non-temporal global stores.
constexpr uint32_t kRawBufferWord3 = 0x00020000u;
constexpr int kStoreSc1 = 16;

// Stores chunk-lane values of one token to its k destination rows, one 1 KiB
// chunk (64 lanes x 16 B) to every row before the next chunk.  Each row gets
// its own buffer resource (base = the row, size = the row), so offsets stay
// 32-bit and anything past the row is dropped by the hardware.
template <int U>
__device__ __forceinline__ void store_rows(const v4u (&v)[U], int rows, int k, int64_t V,
                                           int32_t nch, int lane, v4u *send) {
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int cc = u * kWave + lane;
    if (cc < nch) {
      for (int kk = 0; kk < k; ++kk) {
        const int row = readlane(rows, kk);
        if (row >= 0 && row < V) {
          const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
              send + static_cast<int64_t>(row) * nch, 0, nch * 16, kRawBufferWord3);
          __builtin_amdgcn_raw_buffer_store_b128(v[u], r, cc * 16, 0, kStoreSc1);
        }
      }
    }
  }
}

// Rows of up to 64 * U chunks (H <= 8192): persistent waves, each holding
// one token row in registers while the next token's row is being loaded.
template <int U>
__global__ void __launch_bounds__(kScThreads)
k_scatter(const v4u *__restrict__ x, int64_t T, int32_t k, int32_t nch,
          const int32_t *__restrict__ row_of_slot, const int64_t *n_routed,
          v4u *__restrict__ send) {
  const int lane = lane_id();
  const int64_t V = T * k;
  const int64_t nw = static_cast<int64_t>(gridDim.x) * kScWaves;
  const int64_t gw = static_cast<int64_t>(blockIdx.x) * kScWaves + threadIdx.x / kWave;
  int64_t t = gw;
  if (t < T) {
    v4u v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int cc = u * kWave + lane;
      if (cc < nch) v[u] = __builtin_nontemporal_load(x + t * nch + cc);
    }
    int rows = lane < k ? row_of_slot[t * k + lane] : -1;
    for (;;) {
      const int64_t tn = t + nw;
      v4u w[U];
      int rn = -1;
      if (tn < T) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int cc = u * kWave + lane;
          if (cc < nch) w[u] = __builtin_nontemporal_load(x + tn * nch + cc);
        }
        rn = lane < k ? row_of_slot[tn * k + lane] : -1;
      }
      store_rows<U>(v, rows, k, V, nch, lane, send);
      if (tn >= T) break;
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = w[u];
      rows = rn;
      t = tn;
    }
  }
  // rows after the routed ones (masked slots) are zero-filled
  // a routed count outside [0, V] (not a layout of these slots) fills no row
  const int64_t nr = *n_routed;
  if (nr >= 0 && nr < V) {
    const v4u z = v4u{0u, 0u, 0u, 0u};
    for (int64_t row = nr + gw; row < V; row += nw)
      for (int cc = lane; cc < nch; cc += kWave) send[row * nch + cc] = z;
  }
}

// Longer rows: one wave per token, the row in passes of 1024 chunks.
__global__ void __launch_bounds__(kScThreads)
k_scatter_wide(const v4u *__restrict__ x, int64_t T, int32_t k, int32_t nch,
               const int32_t *__restrict__ row_of_slot, const int64_t *n_routed,
               v4u *__restrict__ send) {
  constexpr int U = 16;
  const int lane = lane_id();
  const int64_t V = T * k;
  const int64_t gw = static_cast<int64_t>(blockIdx.x) * kScWaves + threadIdx.x / kWave;
  const int64_t nw = static_cast<int64_t>(gridDim.x) * kScWaves;
  for (int64_t t = gw; t < T; t += nw) {
    const int rows = lane < k ? row_of_slot[t * k + lane] : -1;
    const v4u *src = x + t * nch;
    for (int c0 = 0; c0 < nch; c0 += U * kWave) {
      v4u v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int cc = c0 + u * kWave + lane;
        if (cc < nch) v[u] = __builtin_nontemporal_load(src + cc);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int cc = c0 + u * kWave + lane;
        if (cc < nch) {
          for (int kk = 0; kk < k; ++kk) {
            const int row = readlane(rows, kk);
            if (row >= 0 && row < V) send[static_cast<int64_t>(row) * nch + cc] = v[u];
          }
        }
      }
    }
  }
  // a routed count outside [0, V] (not a layout of these slots) fills no row
  const int64_t nr = *n_routed;
  if (nr >= 0 && nr < V) {
    const v4u z = v4u{0u, 0u, 0u, 0u};
    for (int64_t row = nr + gw; row < V; row += nw)
      for (int cc = lane; cc < nch; cc += kWave) send[row * nch + cc] = z;
  }
}

hipError_t launch_dispatch_scatter(const uint16_t *x, int64_t T, int32_t k,
                                   int32_t H, const int32_t *row_of_slot,
                                   const int64_t *n_routed, uint16_t *send,
                                   hipStream_t stream) {
  const int32_t nch = H / 8;
  const int64_t need = (T + kScWaves - 1) / kScWaves;
  const dim3 grid(static_cast<unsigned>(need < kScGrid ? (need > 0 ? need : 1) : kScGrid));
  const int per_lane = (nch + kWave - 1) / kWave;
  const v4u *xs = reinterpret_cast<const v4u *>(x);
  v4u *sd = reinterpret_cast<v4u *>(send);
  const dim3 blk(kScThreads);
  if (per_lane <= 1)
    hipLaunchKernelGGL(k_scatter<1>, grid, blk, 0, stream, xs, T, k, nch, row_of_slot, n_routed, sd);
  else if (per_lane <= 2)
    hipLaunchKernelGGL(k_scatter<2>, grid, blk, 0, stream, xs, T, k, nch, row_of_slot, n_routed, sd);
  else if (per_lane <= 4)
    hipLaunchKernelGGL(k_scatter<4>, grid, blk, 0, stream, xs, T, k, nch, row_of_slot, n_routed, sd);
  else if (per_lane <= 8)
    hipLaunchKernelGGL(k_scatter<8>, grid, blk, 0, stream, xs, T, k, nch, row_of_slot, n_routed, sd);
  else if (per_lane <= 14)
    hipLaunchKernelGGL(k_scatter<14>, grid, blk, 0, stream, xs, T, k, nch, row_of_slot, n_routed, sd);
  else if (per_lane <= 16)
    hipLaunchKernelGGL(k_scatter<16>, grid, blk, 0, stream, xs, T, k, nch, row_of_slot, n_routed, sd);
  else
    hipLaunchKernelGGL(k_scatter_wide, grid, blk, 0, stream, xs, T, k, nch, row_of_slot, n_routed, sd);
  return hipGetLastError();
}

}  // namespace uep
