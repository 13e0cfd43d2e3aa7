"""Split-index choice: Algorithm 1 and the evaluation's competitors.

TEST INFRASTRUCTURE ONLY.  The CPU reference for the library's split chooser;
nothing on the product path imports it.  Plain float64 Python, one function
per step of the paper's method, in the paper's order.

A job is a dict with the fields of the library's split-job record: the
per-image output bytes of every split point (``image_bytes[k]``, k = 0 the
input), the server's per-layer forward time for one request
(``srv_layer_s``), the client's per-layer forward time at the training batch
(``cli_layer_s``), the constant and per-byte phase costs of Table 1, the
request layout, the client memory and ``iterations`` (NR_IT).

Sources:
  Design, "Splitting algorithm", Algorithm 1 and the notes after it (split 0
    is costed from the per-iteration time measured while it was profiled).
  Design, "Profiling and modeling runtime", Table 1 (which phase runs where,
    profiled or linear in the split output size) and the concurrency
    paragraph (forward passes of concurrent requests serialise on the
    time-shared GPU, every other phase is parallel, a request waits for the
    wave of requests in front of it).
  Design, "Memory usage estimation" (peak = largest input + output of a layer).
  Evaluation, Methodology, "Competitors" (NoSplit, @Freeze, @Min, NSG) and
    "Training input" (requests of 128 objects, at most 4 run at once).
"""
from __future__ import annotations


class ClientOOM(Exception):
    """The freeze split itself is predicted to exhaust client memory."""


# ------------------------------------------------ Memory usage estimation

def client_memory(job, split):
    """Predicted client GPU bytes when the client continues from ``split``.

    The client holds the received split output, then runs layers
    split+1 .. n_layers; the forward pass peaks at the layer with the largest
    input + output.  The split-independent part (weights, optimiser state,
    training activations) is the caller's ``cli_fixed_mem_bytes``.
    """
    b = job["image_bytes"]
    n = job["n_layers"]
    per_image = b[split]
    for layer in range(split + 1, n + 1):
        per_image = max(per_image, b[layer - 1] + b[layer])
    return job["cli_fixed_mem_bytes"] + job["train_batch"] * per_image


def predicted_oom(job, split):
    cap = job["cli_mem_bytes"]
    return cap > 0 and client_memory(job, split) > cap


# -------------------------------------------- Profiling and modeling runtime

def server_time(job, split):
    """RT_SRV: one iteration's requests on the storage server.

    Per request (Table 1, @server): read the data, read the model, move the
    data to the GPU, forward pass to the split, move the output out of the
    GPU and pickle it (the last two linear in the output bytes).  With the
    split at 0 the server runs no layer, so only reading and pickling the
    input remain.  The training batch arrives as ``train_batch /
    request_images`` requests, at most ``server_slots`` of them at a time: a
    wave's forward passes run one after another on the GPU while everything
    else overlaps, and the next wave waits for this one.
    """
    req_bytes = job["request_images"] * job["image_bytes"][split]
    parallel = job["srv_read_data_s"] + req_bytes * job["srv_pickle_s_per_byte"]
    forward = 0.0
    if split > 0:
        parallel += job["srv_read_model_s"] + job["srv_to_gpu_s"]
        parallel += req_bytes * job["srv_from_gpu_s_per_byte"]
        forward = sum(job["srv_layer_s"][k] for k in range(1, split + 1))
    waiting = job["train_batch"] // job["request_images"]
    total = 0.0
    while waiting > 0:
        in_wave = min(job["server_slots"], waiting)
        total += parallel + in_wave * forward
        waiting -= in_wave
    return total


def network_time(job, split):
    """RT_NW: the iteration's split outputs over the network (profiled bandwidth)."""
    return job["train_batch"] * job["image_bytes"][split] / job["net_bytes_per_s"]


def client_time(job, split):
    """RT_CLI: Table 1, @client: unpickle, build the data loader and copy to the
    GPU (linear in the received bytes), then the forward pass from the split
    to the last profiled layer and the split-independent rest (the layers
    beyond, the backward pass)."""
    received = job["train_batch"] * job["image_bytes"][split]
    linear = received * (job["cli_unpickle_s_per_byte"] + job["cli_loader_s_per_byte"]
                         + job["cli_to_gpu_s_per_byte"])
    forward = sum(job["cli_layer_s"][k] for k in range(split + 1, job["n_layers"] + 1))
    return linear + forward + job["cli_rest_s"]


def epoch_runtime(rt_srv, rt_nw, rt_cli, nr_it):
    """Algorithm 1's per-epoch estimate: the client's work on one iteration
    overlaps the server's work and the transfer of the next."""
    return rt_srv + max(rt_srv + rt_nw, rt_cli) * (nr_it - 1) + rt_cli


# ------------------------------------------------------------- Algorithm 1

def choose_split(job):
    """Runs the three steps of Algorithm 1 and returns
    ``(split_idx, runtimes, earliest)``: the chosen split, the estimate of
    every split the loop costed (a dict, split -> seconds) and the split
    profiled in the second half of epoch 0."""
    freeze_idx = job["freeze_idx"]
    # Right before the first iteration of epoch 0: split at the freeze index;
    # if even that runs out of client memory, the job fails.
    split_idx = freeze_idx
    if predicted_oom(job, split_idx):
        raise ClientOOM(f"split {split_idx} needs {client_memory(job, split_idx)} bytes")
    # Right before the middle iteration: the earliest split that fits.
    split_idx = next(s for s in range(0, freeze_idx + 1) if not predicted_oom(job, s))
    earliest = split_idx
    # End of epoch 0: cost every split in [0, freeze_idx] that fits.
    runtimes = {}
    for potential_split in range(0, freeze_idx + 1):
        if predicted_oom(job, potential_split):
            continue
        if potential_split == 0 and job["nosplit_iter_s"] > 0:
            # split 0 fits, so it was the earliest split and its iteration
            # time was measured during the second half of epoch 0
            runtimes[0] = job["iterations"] * job["nosplit_iter_s"]
            continue
        rt_srv = server_time(job, potential_split)
        rt_cli = client_time(job, potential_split)
        rt_nw = network_time(job, potential_split)
        nr_it = job["iterations"]
        runtimes[potential_split] = epoch_runtime(rt_srv, rt_nw, rt_cli, nr_it)
    split_idx = min(runtimes, key=lambda s: (runtimes[s], s))
    return split_idx, runtimes, earliest


# ------------------------------------------------------------- competitors

def nosplit(job):
    """NoSplit: the whole input goes to the compute tier."""
    return 0


def at_freeze(job):
    """@Freeze: always split at the freezing layer."""
    return job["freeze_idx"]


def at_min(job):
    """@Min: the layer with the smallest output among layers 1..freeze_idx,
    the earliest such layer on ties (split 0 when nothing is frozen)."""
    candidates = range(1, job["freeze_idx"] + 1)
    if not candidates:
        return 0
    return min(candidates, key=lambda k: (job["image_bytes"][k], k))


def nsg(job):
    """NSG (Neurosurgeon's rule with HAPI's estimates): the split that fits in
    client memory with the smallest RT_SRV + RT_NW + RT_CLI, no overlap."""
    best = None
    for s in range(0, job["freeze_idx"] + 1):
        if predicted_oom(job, s):
            continue
        total = server_time(job, s) + network_time(job, s) + client_time(job, s)
        if best is None or total < best[0]:
            best = (total, s)
    if best is None:
        raise ClientOOM("no split in [0, freeze_idx] fits in client memory")
    return best[1]
