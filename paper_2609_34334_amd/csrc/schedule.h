// The paper's collective scheduler on a described multi-node topology.
#pragma once

#include <string>
#include <vector>

namespace hoccl {

struct Topology {
    int G = 0;
    std::vector<int> node;  // NVLink / xGMI domain of each GPU
    std::vector<int> peer;  // symmetric peer of each GPU (-1: none)
    double bw_nvlink = 1.0; // bytes per unit time of an intra-node edge
    double bw_rdma = 1.0;   // bytes per unit time of an inter-node edge
};

struct Schedule {
    std::vector<std::vector<double>> T;                   // expanded traffic
    std::vector<std::vector<std::vector<double>>> stages; // T^1 .. T^n
    std::vector<double> tau;                              // stage durations
    double total = 0.0;                                   // sum of tau
};

std::vector<std::vector<double>> expand_traffic(const Topology &t,
                                                const std::vector<std::vector<double>> &C);
double stage_time(const Topology &t, const std::vector<std::vector<double>> &S);
Schedule decompose(const Topology &t, const std::vector<std::vector<double>> &C);
std::vector<int> interleave_chunks(const std::vector<double> &bytes, double chunk);
std::string schedule_to_json(const Schedule &s);

}  // namespace hoccl
