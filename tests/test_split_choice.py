"""Split-index choice (Algorithm 1, NoSplit, @Freeze, @Min, NSG).

The oracle (``oracle.split``) is pinned against event simulations of the
pipelined iteration loop (Design, "Request flow": requests for the next
iteration go out as the client starts the current one) and of the server's
request waves (Design, "Profiling and modeling runtime": concurrent forward
passes serialise on the GPU, a request waits for the wave in front of it),
against a live-tensor walk of the client's forward pass for the memory
estimate, and against jobs whose answers are fixed by construction.  The
library's ``hapi_choose_split`` is then compared with the oracle on seeded
random jobs over the evaluated models' real per-layer output sizes.
"""
import math

import numpy as np
import pytest

import paper_2210_08650_amd as H
import synth
from oracle import models as OM
from oracle import split as OS

NAMES = ["alexnet", "resnet18", "resnet50", "vgg16", "vit_b16", "densenet_block", "densenet121"]


def _image_bytes(name):
    esz = 4 if name == "alexnet" else 2
    return [e * esz for e in OM.build(name).out_elems()]


def _job(**over):
    j = {"n_layers": 2, "freeze_idx": 2, "train_batch": 128, "request_images": 128,
         "server_slots": 4, "iterations": 100, "image_bytes": [1000, 5000, 10],
         "srv_layer_s": [0.0, 3.0, 1.5], "cli_layer_s": [0.0, 2.0, 2.0],
         "srv_read_data_s": 1.0, "srv_read_model_s": 0.0, "srv_to_gpu_s": 0.0,
         "cli_rest_s": 1.0, "srv_from_gpu_s_per_byte": 0.0, "srv_pickle_s_per_byte": 0.0,
         "cli_unpickle_s_per_byte": 0.0, "cli_loader_s_per_byte": 0.0,
         "cli_to_gpu_s_per_byte": 0.0, "net_bytes_per_s": 128000.0,
         "cli_mem_bytes": 0, "cli_fixed_mem_bytes": 0, "nosplit_iter_s": 0.0}
    j.update(over)
    return j


# ----------------------------------------------------------------- pins

def _simulate_pipeline(rt_srv, rt_nw, rt_cli, iterations):
    """Event walk of the client/server pipeline; returns when the client
    finishes the last iteration.  Iteration 0's requests leave at t = 0; the
    requests of iteration i + 1 leave when the client starts iteration i."""
    send, client_free = 0.0, 0.0
    for _ in range(iterations):
        arrive = send + rt_srv + rt_nw
        start = max(arrive, client_free)
        send = start
        client_free = start + rt_cli
    return client_free


@pytest.mark.parametrize("seed", range(8))
def test_epoch_formula_matches_pipeline_simulation(seed):
    # Algorithm 1's estimate starts the epoch with RT_SRV alone, so the
    # simulated epoch is longer by exactly one transfer (the first iteration's).
    rng = np.random.default_rng(seed)
    for nr_it in (1, 2, 3, 17, 240):
        s, n, c = (float(v) for v in rng.uniform(0.1, 3.0, 3))
        if seed % 2:
            c = s + n + float(rng.uniform(0.1, 1.0))       # client-bound
        sim = _simulate_pipeline(s, n, c, nr_it)
        assert math.isclose(OS.epoch_runtime(s, n, c, nr_it) + n, sim, rel_tol=1e-12)


def _simulate_server(requests, slots, before_gpu, forward, after_gpu):
    """Requests start in waves of ``slots``; in a wave every request does its
    pre-GPU phases at once, then queues for the one GPU (first come, first
    served), then does its post-GPU phases; the next wave starts when the
    last request of this one ends.  Returns (end time, start time of each
    request)."""
    t, starts, left = 0.0, [], requests
    while left:
        wave = min(slots, left)
        gpu_free, ends = t + before_gpu, []
        for _ in range(wave):
            starts.append(t)
            gpu_free += forward
            ends.append(gpu_free + after_gpu)
        t = max(ends)
        left -= wave
    return t, starts


@pytest.mark.parametrize("batch,slots", [(128, 4), (512, 4), (1024, 4), (1536, 4), (3072, 4),
                                         (1024, 1), (1024, 3), (384, 8)])
def test_server_time_matches_request_wave_simulation(batch, slots):
    j = synth.split_job(3, _image_bytes("resnet18"), 8, train_batch=batch, server_slots=slots)
    for split in range(0, 9):
        req_bytes = 128 * j["image_bytes"][split]
        before = j["srv_read_data_s"]
        after = req_bytes * j["srv_pickle_s_per_byte"]
        fwd = 0.0
        if split:
            before += j["srv_read_model_s"] + j["srv_to_gpu_s"]
            after += req_bytes * j["srv_from_gpu_s_per_byte"]
            fwd = float(np.sum(j["srv_layer_s"][1:split + 1]))
        end, starts = _simulate_server(batch // 128, slots, before, fwd, after)
        assert math.isclose(OS.server_time(j, split), end, rel_tol=1e-12), split


def test_server_waits_for_the_wave_in_front():
    # The paper's example: 8 requests, 4 run at once; the last 4 wait exactly
    # as long as the first 4 take.
    j = synth.split_job(4, _image_bytes("resnet50"), 10, train_batch=1024, server_slots=4)
    one_wave = OS.server_time(dict(j, train_batch=512), 10)
    end, starts = _simulate_server(8, 4, 1.0, 0.25, 0.5)
    assert starts[4:] == [end / 2] * 4
    assert math.isclose(OS.server_time(j, 10), 2 * one_wave, rel_tol=1e-12)


def _client_peak_by_walk(image_bytes, split, batch):
    """Live-tensor walk: the received batch is resident; each layer allocates
    its output while its input is alive, then frees the input."""
    live = peak = batch * image_bytes[split]
    for k in range(split + 1, len(image_bytes)):
        live += batch * image_bytes[k]
        peak = max(peak, live)
        live -= batch * image_bytes[k - 1]
    return peak


@pytest.mark.parametrize("name", NAMES)
def test_memory_estimate_matches_live_tensor_walk(name):
    b = _image_bytes(name)
    n = len(b) - 1
    j = synth.split_job(5, b, n, train_batch=256)
    j["cli_fixed_mem_bytes"] = 123_456_789
    mem = [OS.client_memory(j, s) for s in range(n + 1)]
    for s in range(n + 1):
        assert mem[s] == 123_456_789 + _client_peak_by_walk(b, s, 256), s
    # a later split never needs more client memory, so if the freeze split
    # runs out of memory every split does (Algorithm 1's first step)
    assert all(mem[s] >= mem[s + 1] for s in range(n))


def test_hapi_and_nsg_differ_when_overlap_matters():
    # Hand-costed two-layer job (times in seconds, 100 iterations):
    #   split 0: RT_SRV 1,   RT_NW 1,    RT_CLI 5  -> epoch 1 + 5*99 + 5     = 501,    sum 7
    #   split 1: RT_SRV 4,   RT_NW 5,    RT_CLI 3  -> epoch 4 + 9*99 + 3     = 898,    sum 12
    #   split 2: RT_SRV 5.5, RT_NW 0.01, RT_CLI 1  -> epoch 5.5 + 5.51*99 + 1 = 551.99, sum 6.51
    # Overlap hides the client's work at split 0, so Algorithm 1 keeps it;
    # the plain sum (NSG) prefers the small transfer at split 2.
    j = _job(srv_read_model_s=0.0)
    split, runtimes, earliest = OS.choose_split(j)
    assert (split, earliest, OS.nsg(j), OS.at_min(j), OS.at_freeze(j)) == (0, 0, 2, 2, 2)
    assert [round(runtimes[s], 9) for s in range(3)] == [501.0, 898.0, 551.99]
    # client memory 128 * max(in + out): 768000, 641280, 1280 bytes; a 700 kB
    # client cannot take split 0, so the earliest profiled split is 1 and the
    # choice moves to split 2
    j = _job(cli_mem_bytes=700_000)
    split, runtimes, earliest = OS.choose_split(j)
    assert (split, earliest, sorted(runtimes)) == (2, 1, [1, 2])
    assert OS.nsg(j) == 2
    with pytest.raises(OS.ClientOOM):
        OS.choose_split(_job(cli_mem_bytes=1279))


def test_ties_take_the_earliest_split():
    flat = _job(image_bytes=[7, 7, 7], srv_layer_s=[0.0, 0.0, 0.0], cli_layer_s=[0.0, 0.0, 0.0],
                srv_read_data_s=0.0, net_bytes_per_s=1e300)
    split, runtimes, _ = OS.choose_split(flat)
    assert split == 0 and len(set(runtimes.values())) == 1
    assert OS.at_min(flat) == 1 and OS.nsg(flat) == 0
    assert OS.at_min(_job(freeze_idx=0)) == 0


def test_nosplit_uses_its_measured_iteration_time():
    j = _job(nosplit_iter_s=2.0)
    split, runtimes, _ = OS.choose_split(j)
    assert runtimes[0] == 200.0 and split == 0
    split, runtimes, _ = OS.choose_split(_job(nosplit_iter_s=6.0))
    assert runtimes[0] == 600.0 and split == 2


def test_transformer_min_split_is_layer_one():
    # Evaluation, vs static splitting: @Min splits the Transformer at layer 1.
    b = _image_bytes("vit_b16")
    assert OS.at_min(synth.split_job(6, b, len(b) - 1)) == 1


# ------------------------------------------------- library vs the oracle

def _oracle_all(j):
    split, runtimes, earliest = OS.choose_split(j)
    return split, runtimes, earliest


def _assert_same_argmin(got, want, values):
    if got != want:  # only an exact or rounding-level tie may differ
        assert math.isclose(values[got], values[want], rel_tol=1e-12), (got, want)
        assert want < got


@pytest.mark.parametrize("name", NAMES)
@pytest.mark.parametrize("batch", [128, 512, 1536, 3072])
def test_library_matches_oracle(name, batch):
    b = _image_bytes(name)
    n = len(b) - 1
    for seed in range(6):
        freeze = n if seed % 3 == 0 else int(np.random.default_rng(seed).integers(0, n + 1))
        j = synth.split_job(10 + seed, b, freeze, train_batch=batch)
        if seed % 2:
            # a client that fits only the later splits
            io = sorted(batch * (b[k - 1] + b[k]) for k in range(1, n + 1))
            j["cli_mem_bytes"] = int(io[len(io) // 2]) + batch * max(b)
            j["cli_fixed_mem_bytes"] = batch * max(b) // 2
        if seed == 4:
            j["nosplit_iter_s"] = 1.5
        try:
            want = _oracle_all(j)
        except OS.ClientOOM:
            with pytest.raises(H.HapiError) as e:
                H.hapi_choose_split(**j)
            assert e.value.code == H.HAPI_E_NOMEM
            continue
        choice, est = H.hapi_choose_split(**j)
        assert len(est) == freeze + 1
        for s, e in enumerate(est):
            assert e["cli_mem_bytes"] == OS.client_memory(j, s)
            assert e["oom"] == int(OS.predicted_oom(j, s))
            for key, fn in (("rt_srv", OS.server_time), ("rt_nw", OS.network_time),
                            ("rt_cli", OS.client_time)):
                assert math.isclose(e[key], fn(j, s), rel_tol=1e-12), (s, key)
            if s in want[1]:
                assert math.isclose(e["epoch_s"], want[1][s], rel_tol=1e-12), s
        _assert_same_argmin(choice["hapi"], want[0], {s: est[s]["epoch_s"] for s in want[1]})
        assert choice["earliest"] == want[2]
        sums = {s: est[s]["sum_s"] for s in range(freeze + 1) if not est[s]["oom"]}
        _assert_same_argmin(choice["nsg"], OS.nsg(j), sums)
        assert choice["freeze"] == OS.at_freeze(j) == freeze
        assert choice["min_output"] == OS.at_min(j)
        assert choice["nosplit"] == OS.nosplit(j) == 0


def test_library_validation():
    def code(**over):
        with pytest.raises(H.HapiError) as e:
            H.hapi_choose_split(**_job(**over))
        return e.value.code
    assert code(freeze_idx=3) == H.HAPI_E_INVAL
    assert code(freeze_idx=-1) == H.HAPI_E_INVAL
    assert code(train_batch=200) == H.HAPI_E_INVAL        # not a multiple of 128
    assert code(server_slots=0) == H.HAPI_E_INVAL
    assert code(iterations=0) == H.HAPI_E_INVAL
    assert code(srv_layer_s=[0.0, -1.0, 1.0]) == H.HAPI_E_INVAL
    assert code(cli_layer_s=[0.0, float("nan"), 1.0]) == H.HAPI_E_INVAL
    assert code(net_bytes_per_s=0.0) == H.HAPI_E_INVAL
    assert code(image_bytes=[1000, 0, 10]) == H.HAPI_E_INVAL
    assert code(image_bytes=[1000, 2**62, 2**62]) == H.HAPI_E_INVAL  # in + out overflows
    assert code(reserved0=1) == H.HAPI_E_INVAL
    assert code(cli_mem_bytes=1279) == H.HAPI_E_NOMEM
    with pytest.raises(ValueError):
        H.hapi_choose_split(**_job(image_bytes=[1, 2]))
    j = _job()
    del j["cli_layer_s"]
    with pytest.raises(H.HapiError):
        H.hapi_choose_split(**j)
    choice, est = H.hapi_choose_split(**_job(cli_mem_bytes=1280))
    assert choice == {"hapi": 2, "earliest": 2, "freeze": 2, "min_output": 2, "nosplit": 0,
                      "nsg": 2}
    assert [e["oom"] for e in est] == [1, 1, 0]
