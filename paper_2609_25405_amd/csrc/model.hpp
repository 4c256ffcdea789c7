// The host-side model handle behind orthrus_model: configuration, weight pointers, and the
// per-handle state of the step (metadata staging, kernel timing).
#pragma once

#include <hip/hip_runtime.h>

#include <mutex>
#include <string>
#include <vector>

#include "plan.hpp"

struct orthrus_model : public orthrus::Model {
    // pinned host staging for the per-step metadata upload, double-buffered with events:
    // fine-grained (coherent) host memory that the upload kernel reads through its device
    // address; buffers outgrown by a larger batch are retired, not freed, until the handle is
    // destroyed
    std::mutex mu;
    void *stage[2] = {nullptr, nullptr};
    void *stage_dev[2] = {nullptr, nullptr};
    size_t stage_bytes[2] = {0, 0};
    std::vector<void *> retired;
    hipEvent_t ev[2] = {nullptr, nullptr};
    int next = 0;
    // steps with two row groups (two models) run the generator group's launches on `aux`
    // (default priority), forked from the step's stream after the plan upload and joined to it
    // before the final norm; step_mu serialises the host side of such steps on this handle
    hipStream_t aux = nullptr;
    hipEvent_t ev_fork = nullptr, ev_join = nullptr;
    std::mutex step_mu;
    // kernel timing (orthrus_profile_begin / _end); prof_only (orthrus_profile_only) limits the
    // timed launches to one name, empty = all
    bool profiling = false;
    std::string prof_only;
    struct Mark { int name; hipEvent_t a, b; };
    std::vector<std::string> prof_names;
    std::vector<Mark> marks;
};
