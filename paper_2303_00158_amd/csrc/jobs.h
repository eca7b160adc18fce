// Jobs: the body of a kernel as a value that knows how to run one logical
// workgroup, so that one launch can serve two independent pieces of work.
//
// A job type J has `__device__ void run(int64_t blk, int64_t nblk) const`,
// which does the work of logical workgroup blk out of nblk (256 threads).
// job2_kernel gives the first workgroups of the grid to one job and the
// rest to another.  Merging independent steps this way saves a launch and
// lets the latencies of the two overlap; every job runs with the launch
// bounds of 256 threads, and the LDS of both is reserved.
#pragma once

#include "internal.h"

namespace gnn {

template <class J>
__global__ void __launch_bounds__(256) job_kernel(J j) {
    j.run(blockIdx.x, gridDim.x);
}

// Workgroups [0, na) run a, [na_pad, grid) run b; na_pad (a multiple of 8)
// keeps b's logical workgroup index congruent to its physical one modulo the
// XCD count, which jobs that map work to XCDs rely on.
template <class A, class B>
__global__ void __launch_bounds__(256) job2_kernel(A a, unsigned na, unsigned na_pad, B b) {
    if (blockIdx.x < na_pad) {
        if (blockIdx.x < na) a.run(blockIdx.x, na);
    } else {
        b.run(blockIdx.x - na_pad, gridDim.x - na_pad);
    }
}

// Any number of roles in one launch: Pack<J0, J1, ...> gives each role a
// range of workgroups, every range but the last padded to a multiple of 8
// (as in job2_kernel).  A role with zero workgroups takes none.
template <class... J> struct Pack;
template <> struct Pack<> {
    __device__ void run(unsigned) const {}
    unsigned grid() const { return 0; }
};
template <class J, class... R> struct Pack<J, R...> {
    J j;
    unsigned n, npad;
    Pack<R...> rest;
    __device__ void run(unsigned b) const {
        if (b < npad) {
            if (b < n) j.run(b, n);
        } else {
            rest.run(b - npad);
        }
    }
    unsigned grid() const {
        const unsigned g = rest.grid();
        return g == 0 ? n : npad + g;  // the last non-empty role needs no padding
    }
};

// A role of a packed launch: a job and its workgroup count.
template <class J> struct Role {
    J j;
    unsigned n;
};
template <class J> Role<J> role(const J &j, unsigned n) { return Role<J>{j, n}; }

inline Pack<> make_pack() { return Pack<>{}; }
template <class J, class... R> Pack<J, R...> make_pack(const Role<J> &r, const Role<R> &...rest) {
    Pack<J, R...> p;
    p.j = r.j;
    p.n = r.n;
    p.npad = (r.n + 7) / 8 * 8;
    p.rest = make_pack(rest...);
    return p;
}

// The same job for up to kMaxCopies independent instances (for example the
// same sampling phase of several training steps): copy c takes workgroups
// [c * npad, c * npad + n), npad = n rounded up to a multiple of 8 (as in a
// Pack, so each copy's logical index stays congruent to its physical one
// modulo the XCD count).  The copy index is uniform per workgroup.
constexpr int kMaxCopies = 4;
template <class J> struct Multi {
    J j[kMaxCopies];
    int g;
    unsigned n, npad;
    __device__ void run(int64_t b, int64_t) const {
        const int c = static_cast<int>(b / npad);
        const int64_t lb = b - static_cast<int64_t>(c) * npad;
        if (c < g && lb < n) j[c].run(lb, n);
    }
};
// make(c) gives copy c's job; g copies of n workgroups each.
template <class Make> auto multi_role(Make &&make, int g, unsigned n) {
    using J = decltype(make(0));
    Multi<J> m{};
    for (int c = 0; c < g; ++c) m.j[c] = make(c);
    m.g = g;
    m.n = n;
    m.npad = (n + 7) / 8 * 8;
    return Role<Multi<J>>{m, n ? m.npad * static_cast<unsigned>(g) : 0u};
}

template <class P>
__global__ void __launch_bounds__(256) pack_kernel(P p) {
    p.run(blockIdx.x);
}

template <class J>
gnn_status launch_job(const J &j, unsigned grid, hipStream_t s, const char *what) {
    if (grid == 0) return GNN_OK;
    job_kernel<J><<<grid, 256, 0, s>>>(j);
    return launch_status(what);
}

template <class A, class B>
gnn_status launch_job2(const A &a, unsigned na, const B &b, unsigned nb, hipStream_t s, const char *what) {
    if (na == 0) return launch_job(b, nb, s, what);
    if (nb == 0) return launch_job(a, na, s, what);
    const unsigned pad = (na + 7) / 8 * 8;
    job2_kernel<A, B><<<pad + nb, 256, 0, s>>>(a, na, pad, b);
    return launch_status(what);
}

// Launches the roles together (in one kernel) on s.
template <class... J>
gnn_status launch_jobs(hipStream_t s, const char *what, const Role<J> &...roles) {
    const auto p = make_pack(roles...);
    static_assert(sizeof(p) <= 4096, "kernel arguments of a packed launch exceed 4 KiB");
    const unsigned grid = p.grid();
    if (grid == 0) return GNN_OK;
    pack_kernel<decltype(p)><<<grid, 256, 0, s>>>(p);
    return launch_status(what);
}

}  // namespace gnn
