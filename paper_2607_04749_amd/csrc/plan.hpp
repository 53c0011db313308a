// plan.hpp -- host planner entry points (plan.hip).
#pragma once

#include <stdexcept>
#include <string>
#include <vector>

#include "etc_internal.hpp"

namespace etc {

struct PlanError : std::runtime_error {
  PlanError(int c, std::string m);
  int code;
};

std::vector<LogicalTensor> build_tensor_table(const etc_model_desc& m);
int stage_of(const LogicalTensor& t, int role, const Grid& g, int num_layers);
RankLayout build_layout(const std::vector<LogicalTensor>& T, const Grid& g, int num_layers, int rank);

// throws PlanError on bad input
void validate(const etc_model_desc& m, const etc_parallel_cfg& src, const etc_parallel_cfg& dst);
// per-tensor routing records (stages per copy role, single-copy flag)
void build_route_tensors(etc_plan_t& P);
// routing context of a plan's host tables
RouteCtx host_route_ctx(const etc_plan_t& P);
// COST of one replica pair on the host (rows: a replica's target ranks)
std::vector<uint64_t> host_replica_cost(const etc_plan_t& P);
// the migration sketch, replica by replica, into P.home (dead: failed sources)
void sketch_pairing(etc_plan_t& P, const std::vector<char>& dead);
// layouts, routing, message layouts (host only); P.home must be set
void build_host_plan(etc_plan_t& P);
// virtual rank allocator (defrag.hip); returns an ETC_ status
int defrag(int S, int D, const int32_t* home, const std::vector<char>& dead, int mode,
           int32_t* placement, int32_t* ops, int* nops);
// migration sketch (sketch.hip): pair[i] = column paired with row i, or -1
uint64_t solve_sketch(const uint64_t* cost, int M, int N, int32_t* pair);
// copy descriptors of one rank (terminated by a sentinel box holding the tile count)
std::vector<CopyBox> build_pack_boxes(const etc_plan_t& P, int s, std::vector<int32_t>* peers,
                                      uint64_t* bytes);
std::vector<CopyBox> build_unpack_boxes(const etc_plan_t& P, int d, std::vector<int32_t>* peers,
                                        uint64_t* bytes);
// Refer boxes of target d: its paired source's arenas -> its arenas
std::vector<CopyBox> build_refer_boxes(const etc_plan_t& P, int d, uint64_t* bytes);

}  // namespace etc
