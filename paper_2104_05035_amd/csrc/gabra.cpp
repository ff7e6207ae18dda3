// GABRA: genetic-algorithm allocation of network partitions to GPUs
// (model-parallelisation section of the paper, "Genetic Algorithm Based
// Resource Allocation"; eqs. 3-10, Algorithms 1-3).  Host code only: it
// decides where the partitions of a model-parallel split run, before any
// kernel is launched.
//
// Problem: partition i has computation load p_i, GPU j capacity d_j; running
// i on j earns c_ij = p_i / d_j (eq. 3).  An allocation assigns every
// partition to exactly one GPU (eq. 9) without exceeding any GPU's capacity
// (eq. 8) and maximises the total profit (eq. 7).  Optionally (the paper's
// stated assumption) every GPU must run at least one partition.
//
// Representation and operators, with the readings taken where the paper is
// garbled or silent:
//   chromosome   gene i = GPU of partition i (eq. 9 holds by construction);
//                fitness = total profit of the allocation;
//   population   drawn partition by partition, each to a GPU chosen
//                uniformly among those with room left; a stuck chromosome is
//                redrawn (Algorithm 2);
//   selection    two independent roulette-wheel spins, probability
//                fitness / total fitness;
//   crossover    with probability 0.8: cut at half the length (Algorithm 3);
//                offspring 1 = first half of Y1 + second half of Y2,
//                offspring 2 = first half of Y2 + second half of Y1 (genes keep
//                their positions); one of the two by a fair draw; otherwise a
//                copy of Y1;
//   mutation     inversion of a segment [a, b], a < b uniform over all pairs;
//   acceptance   an offspring equal to a population member, or infeasible, is
//                dropped and selection starts over (not counted as a
//                generation; a bound on all attempts guarantees termination);
//                otherwise it replaces the worst member (first on ties), and
//                becomes the best-so-far when strictly fitter.
// Random numbers: SplitMix64 (Steele, Lea, Flood, OOPSLA 2014), draw k of
// seed s = mix(s + (k+1) * 0x9E3779B97F4A7C15); doubles from the top 53 bits.
#include <cmath>
#include <cstdint>
#include <vector>

#include "kernels.hpp"

namespace {

class SplitMix64 {
  public:
    explicit SplitMix64(uint64_t seed) : s_(seed) {}
    uint64_t next() {
        s_ += 0x9E3779B97F4A7C15ull;
        uint64_t z = s_;
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        return z ^ (z >> 31);
    }
    double uniform() { return (double)(next() >> 11) * (1.0 / 9007199254740992.0); }
    int below(int n) {
        const int k = (int)(uniform() * n);
        return k < n - 1 ? k : n - 1;
    }

  private:
    uint64_t s_;
};

using Chromo = std::vector<int>;

struct Problem {
    int n, m;
    const double* p;
    const double* d;
    bool every_gpu;
    std::vector<double> c;  // c[i * m + j] = p_i / d_j

    bool feasible(const Chromo& b) const {
        std::vector<double> load(m, 0.0);
        for (int i = 0; i < n; ++i) load[b[i]] += p[i];
        for (int j = 0; j < m; ++j)
            if (load[j] > d[j]) return false;
        if (every_gpu) {
            std::vector<char> used(m, 0);
            for (int i = 0; i < n; ++i) used[b[i]] = 1;
            for (int j = 0; j < m; ++j)
                if (!used[j]) return false;
        }
        return true;
    }
    double fitness(const Chromo& b) const {
        double f = 0.0;
        for (int i = 0; i < n; ++i) f += c[(size_t)i * m + b[i]];
        return f;
    }
};

// One chromosome of the initial population; false if every try got stuck.
bool draw_initial(const Problem& pr, SplitMix64& rng, int tries, Chromo& out) {
    std::vector<double> rem(pr.m);
    std::vector<int> fits;
    fits.reserve(pr.m);
    for (int t = 0; t < tries; ++t) {
        for (int j = 0; j < pr.m; ++j) rem[j] = pr.d[j];
        out.clear();
        bool stuck = false;
        for (int i = 0; i < pr.n && !stuck; ++i) {
            fits.clear();
            for (int j = 0; j < pr.m; ++j)
                if (pr.p[i] <= rem[j]) fits.push_back(j);
            if (fits.empty()) {
                stuck = true;
                break;
            }
            const int j = fits[rng.below((int)fits.size())];
            rem[j] -= pr.p[i];
            out.push_back(j);
        }
        if (!stuck && pr.feasible(out)) return true;
    }
    return false;
}

int roulette(const std::vector<double>& f, SplitMix64& rng) {
    double total = 0.0;
    for (double v : f) total += v;
    const double r = rng.uniform() * total;
    double acc = 0.0;
    for (size_t k = 0; k < f.size(); ++k) {
        acc += f[k];
        if (r < acc) return (int)k;
    }
    return (int)f.size() - 1;
}

}  // namespace

using namespace rat3d;

extern "C" {

rat3d_status rat3d_gabra(int n, const double* loads, int m, const double* capacities,
                         const rat3d_gabra_params* params, int32_t* assignment, double* profit,
                         rat3d_gabra_stats* stats) {
    if (n < 1 || m < 1 || !loads || !capacities || !params || !assignment || !profit) {
        set_error("rat3d_gabra: n, m must be >= 1 and loads, capacities, params, assignment, "
                  "profit non-NULL");
        return RAT3D_EINVAL;
    }
    for (int i = 0; i < n; ++i)
        if (!(loads[i] > 0.0) || !std::isfinite(loads[i])) {
            set_error("rat3d_gabra: load %d is not a positive finite number", i);
            return RAT3D_EINVAL;
        }
    for (int j = 0; j < m; ++j)
        if (!(capacities[j] > 0.0) || !std::isfinite(capacities[j])) {
            set_error("rat3d_gabra: capacity %d is not a positive finite number", j);
            return RAT3D_EINVAL;
        }
    const rat3d_gabra_params& q = *params;
    if (q.population < 2 || q.generations < 0 || !(q.crossover_p >= 0.0 && q.crossover_p <= 1.0) ||
        q.max_attempts < 0 || q.init_tries < 0) {
        set_error("rat3d_gabra: needs population >= 2, generations >= 0, crossover_p in [0, 1], "
                  "max_attempts >= 0, init_tries >= 0");
        return RAT3D_EINVAL;
    }
    Problem pr{n, m, loads, capacities, q.every_gpu != 0, std::vector<double>((size_t)n * m)};
    for (int i = 0; i < n; ++i)
        for (int j = 0; j < m; ++j) pr.c[(size_t)i * m + j] = loads[i] / capacities[j];
    const int64_t max_attempts = q.max_attempts > 0 ? q.max_attempts : 50 * (int64_t)q.generations;
    const int tries = q.init_tries > 0 ? q.init_tries : 1000;

    SplitMix64 rng(q.seed);
    std::vector<Chromo> pop(q.population);
    std::vector<double> fit(q.population);
    for (int k = 0; k < q.population; ++k) {
        if (!draw_initial(pr, rng, tries, pop[k])) {
            set_error("rat3d_gabra: no feasible allocation found for the initial population "
                      "(%d tries)", tries);
            return RAT3D_EINVAL;
        }
        fit[k] = pr.fitness(pop[k]);
    }
    int best = 0;
    for (int k = 1; k < q.population; ++k)
        if (fit[k] > fit[best]) best = k;
    Chromo Z = pop[best];
    double fZ = fit[best];

    int64_t t = 0, attempts = 0, dups = 0, infeas = 0;
    Chromo w(n);
    while (t < q.generations && attempts < max_attempts) {
        ++attempts;
        const Chromo& y1 = pop[roulette(fit, rng)];
        const Chromo& y2 = pop[roulette(fit, rng)];
        if (rng.uniform() < q.crossover_p) {
            const int cp = n / 2;
            const bool first = rng.uniform() < 0.5;
            const Chromo& head = first ? y1 : y2;
            const Chromo& tail = first ? y2 : y1;
            for (int i = 0; i < n; ++i) w[i] = i < cp ? head[i] : tail[i];
        } else {
            w = y1;
        }
        if (n >= 2) {
            int a = rng.below(n), b = rng.below(n - 1);
            if (b >= a) ++b;
            if (a > b) std::swap(a, b);
            for (; a < b; ++a, --b) std::swap(w[a], w[b]);
        }
        bool dup = false;
        for (const Chromo& z : pop)
            if (z == w) {
                dup = true;
                break;
            }
        if (dup) {
            ++dups;
            continue;
        }
        if (!pr.feasible(w)) {
            ++infeas;
            continue;
        }
        const double fw = pr.fitness(w);
        int worst = 0;
        for (int k = 1; k < q.population; ++k)
            if (fit[k] < fit[worst]) worst = k;
        pop[worst] = w;
        fit[worst] = fw;
        if (fw > fZ) {
            Z = w;
            fZ = fw;
        }
        ++t;
    }
    for (int i = 0; i < n; ++i) assignment[i] = Z[i];
    *profit = fZ;
    if (stats) {
        stats->generations = t;
        stats->duplicates = dups;
        stats->infeasible = infeas;
        stats->attempts = attempts;
    }
    return RAT3D_OK;
}

}  // extern "C"
