"""Batched layer chains over the libspyke entry points.

A :class:`Chain` owns every device buffer of one batch (allocated once, at
construction) and runs a workload's stages as a fixed sequence of C-ABI
calls on one stream, with no host synchronisation and no allocation inside
:meth:`Chain.forward` / :meth:`Chain.learn`:

* source: ``spk_encode_latency`` (images + filter bank) or a given wave;
  with ``local_norm=(radius, eps)`` the filter map is locally normalised
  (``spk_local_normalization``) before ``spk_rank_latency`` codes it;
* each conv stage: ``spk_conv_fire`` then ``spk_kwta`` (the winners feed
  plasticity and, for the last layer, the decision; in :meth:`Chain.step`
  the kWTA of a layer whose plasticity starts early runs on that layer's
  side stream, ahead of its plasticity); when its input is the
  encoder's or a pool's output, whose wave is Eq.1 of its first-spike map by
  construction, ``spk_conv_fire_first_spike`` reads that map instead of the
  T planes of the wave;
* with ``fused=True``, a conv stage with a finite threshold and stride 1 whose
  input is a first-spike map, followed by a pool stage with window = stride
  and no padding, runs as one ``spk_conv_fire_pool`` launch (conv, fire and
  the first-spike pooling fused) that fills both stages' buffers;
* each pool stage: ``spk_pool_first_spike`` on the first-spike map of the
  stage below (which equals ``spk_pool`` on its wave whenever that wave is
  cumulative -- always the case for non-negative weights), or ``spk_pool``
  on the wave when constructed with ``pool_from_first_spike=False``;
* with ``want_waves=False`` no Eq.1 wave is written where a first-spike map
  carries the same information: the encoder and the pools write first-spike
  maps only, and a layer whose input is such a map learns from it
  (``spk_stdp_first_spike`` / ``spk_rstdp_first_spike``); only a conv stage
  fed by another conv still writes per-step spikes;
* after a reward-modulated last layer: ``spk_decide``;
* learning: ``spk_stdp`` / ``spk_rstdp`` per conv stage (frozen forward,
  ordered replay within the batch).  The layers' updates touch disjoint
  weights, so with ``concurrent_learn`` they run on side streams (default
  priority) that fork from and join back into the caller's stream; in
  :meth:`Chain.step` the layers up to the second-to-last conv stage fork right
  after that stage's kWTA, overlapping the rest of the forward.

A stage list is any sequence of objects with the attributes of
``Conv(cin, cout, K, pad, thr, k, r, learn, a_plus, a_minus, lb, ub,
stabilizer)`` (and optionally ``stride``, default 1: a strided stage calls
the ``*_strided`` entry points) and ``Pool(P, R, D)``.
"""
from __future__ import annotations

import copy
import math

import torch

from . import (pool_out_size, conv_out_size, spk_conv_fire, spk_conv_fire_first_spike, spk_conv_fire_workspace_size,
               spk_conv_fire_strided, spk_conv_fire_first_spike_strided, spk_conv_fire_strided_workspace_size,
               spk_conv_fire_pool,
               spk_rstdp_strided, spk_stdp_strided, spk_stdp_first_spike, spk_rstdp_first_spike, spk_decide,
               spk_encode_latency, spk_encode_latency_workspace_size, spk_kwta, spk_kwta_workspace_size,
               spk_local_normalization, spk_pool, spk_pool_first_spike, spk_rank_latency, spk_rstdp, spk_stdp,
               spk_stdp_workspace_size)


def _is_conv(st):
    return hasattr(st, "cout")


def _stride(st):
    return getattr(st, "stride", 1)


class Chain:
    def __init__(self, stages, B, T, H, W, cin, source="image", filter_bank=None, filter_threshold=0.0,
                 n_classes=10, device="cuda", want_potentials=True, pool_from_first_spike=True,
                 concurrent_learn=True, want_spikes=True, local_norm=None, fused=False, want_waves=True):
        self.stages = [copy.copy(st) for st in stages]  # own copies: set_rates changes them
        self.fused = fused
        # without waves, the encoder's and the pools' outputs are first-spike maps only
        self.want_waves = want_waves or source != "image"
        self.pool_from_first_spike = pool_from_first_spike
        self.B, self.T, self.source = B, T, source
        self.n_classes = n_classes
        self.filter_threshold = filter_threshold
        dev = torch.device(device)
        u8, f32, i32 = torch.uint8, torch.float32, torch.int32
        ws_bytes = 0
        if source == "image":
            self.bank = filter_bank.to(dev).contiguous()
            C = self.bank.shape[0]
            self.image = torch.zeros((B, H, W), dtype=u8, device=dev)
            ws_bytes = max(ws_bytes, spk_encode_latency_workspace_size(B, C, H, W, T))
            # local_norm = (radius, eps): filter, spk_local_normalization, then the rank-order code
            self.local_norm = local_norm
            if local_norm is not None:
                self.inten = torch.empty((B, C, H, W), dtype=f32, device=dev)
                self.inten_norm = torch.empty((B, C, H, W), dtype=f32, device=dev)
        else:
            C = cin
            self.image = None
            self.local_norm = None
        self.input_wave = torch.zeros((B, T, C, H, W), dtype=u8, device=dev) if self.want_waves else None
        self.input_tf = torch.zeros((B, C, H, W), dtype=u8, device=dev) if source == "image" else None
        self.bufs = []
        c, h, w = C, H, W
        for si, st in enumerate(self.stages):
            b = {}
            if _is_conv(st):
                assert st.cin == c, "stage input channels do not match"
                ho, wo = conv_out_size(h, st.K, st.pad, _stride(st)), conv_out_size(w, st.K, st.pad, _stride(st))
                b["P"] = torch.empty((B, T, st.cout, ho, wo), dtype=f32, device=dev) if want_potentials else False
                # without want_spikes a conv stage's per-step spikes are written only when the next
                # stage reads them (a conv, or a pool on waves); the first-spike map always is
                nxt = self.stages[si + 1] if si + 1 < len(self.stages) else None
                spikes_read = nxt is not None and (_is_conv(nxt) or not pool_from_first_spike)
                b["S"] = (torch.empty((B, T, st.cout, ho, wo), dtype=u8, device=dev) if want_spikes or spikes_read
                          else False)
                b["tf"] = torch.empty((B, st.cout, ho, wo), dtype=u8, device=dev)
                b["vf"] = torch.empty((B, st.cout, ho, wo), dtype=f32, device=dev)
                b["win"] = torch.empty((B, st.k, 4), dtype=i32, device=dev)
                b["nw"] = torch.empty((B,), dtype=i32, device=dev)
                b["weight"] = torch.empty((st.cout, st.cin, st.K, st.K), dtype=f32, device=dev)
                # each learning layer has its own plasticity workspace (the layers update concurrently)
                b["ws_learn"] = (torch.empty(max(256, spk_stdp_workspace_size(st.cout, st.cin, st.K, B, st.k)),
                                             dtype=u8, device=dev) if st.learn is not None else None)
                b["ws_kwta"] = (torch.empty(max(256, spk_kwta_workspace_size(B, st.cout, ho, wo)), dtype=u8,
                                            device=dev) if st.learn is not None else None)
                ws_bytes = max(ws_bytes,
                               spk_conv_fire_strided_workspace_size(B, T, st.cin, h, w, st.cout, st.K, _stride(st),
                                                                    st.pad),
                               spk_kwta_workspace_size(B, st.cout, ho, wo))
                c, h, w = st.cout, ho, wo
            else:
                ho, wo = pool_out_size(h, st.P, st.R, st.D), pool_out_size(w, st.P, st.R, st.D)
                b["out"] = torch.empty((B, T, c, ho, wo), dtype=u8, device=dev) if self.want_waves else False
                b["out_tf"] = torch.empty((B, c, ho, wo), dtype=u8, device=dev)
                h, w = ho, wo
            b["shape_in"] = None
            self.bufs.append(b)
        self.workspace = torch.empty(max(ws_bytes, 256), dtype=u8, device=dev)
        self.labels = torch.zeros((B,), dtype=i32, device=dev)
        self.decision = torch.empty((B,), dtype=i32, device=dev)
        self.reward = torch.zeros((B,), dtype=torch.int8, device=dev)
        self.pre_waves = [None] * len(self.stages)
        self.pre_tf = [None] * len(self.stages)  # a conv stage's input first-spike map, when it has one
        n_learn = sum(1 for st in self.stages if _is_conv(st) and st.learn is not None)
        self.concurrent_learn = concurrent_learn and n_learn > 1
        if self.concurrent_learn:
            self._side = [torch.cuda.Stream(device=dev) for _ in range(n_learn)]
            self._forks = [torch.cuda.Event(), torch.cuda.Event()]
            self._joins = [torch.cuda.Event() for _ in range(n_learn)]
        # With concurrent learning, the layers up to the second-to-last conv stage
        # start their plasticity right after that stage's kWTA (their inputs and
        # winners are final then, and no later stage reads their weights), so it
        # overlaps the rest of the forward; the last conv stage's follows it.
        convs = [i for i, st in enumerate(self.stages) if _is_conv(st)]
        self._early_at = convs[-2] if self.concurrent_learn and len(convs) >= 2 else None
        # ... and in a step the kWTA of those layers runs on their side stream too, ahead of
        # their plasticity (its winners feed nothing else), overlapping the next stages
        self._side_kwta = {i: j for j, (i, st, b) in enumerate(self._learners())
                           if self._early_at is not None and i <= self._early_at}
        self._conv_done = {i: torch.cuda.Event() for i in self._side_kwta}
        self._launched = set()
        # step(defer_learn=True): learner stage -> its join event, waited for by the next
        # forward right before the stage that rewrites the learner's input
        self._pending = {}

    # ---------------------------------------------------------------- setup
    def conv_stages(self):
        return [i for i, st in enumerate(self.stages) if _is_conv(st)]

    def set_weights(self, weights):
        for i, wt in zip(self.conv_stages(), weights):
            self.bufs[i]["weight"].copy_(wt)

    def weights(self):
        return [self.bufs[i]["weight"] for i in self.conv_stages()]

    def set_rates(self, layer, a_plus, a_minus):
        """Learning rates of conv layer `layer` (0-based among the conv stages)
        for the steps enqueued from now on: a schedule (the tutorial's adaptive
        or multiplied rates) is a sequence of such calls between steps."""
        st = self.stages[self.conv_stages()[layer]]
        st.a_plus, st.a_minus = float(a_plus), float(a_minus)

    def rates(self, layer):
        st = self.stages[self.conv_stages()[layer]]
        return st.a_plus, st.a_minus

    def set_input(self, image=None, wave=None, labels=None):
        if image is not None:
            self.image.copy_(image)
        if wave is not None:
            self.input_wave.copy_(wave)
        if labels is not None:
            self.labels.copy_(labels)

    # ---------------------------------------------------------------- run
    def forward(self, stream=None, hook=None, early_learn=False):
        """Enqueue the forward of the batch.  hook(name, phase), if given, is
        called right before (phase 0) and after (phase 1) each C-ABI call;
        names are "encode", "conv<i>", "kwta<i>", "pool<i>", "decide"."""
        mark = hook or (lambda name, phase: None)
        main = stream if stream is not None else torch.cuda.current_stream()
        self._wait_pending(-1, main)
        if self.source == "image":
            mark("encode", 0)
            wave_out = self.input_wave if self.want_waves else False
            if self.local_norm is None:
                spk_encode_latency(self.image, self.bank, self.T, self.filter_threshold, wave=wave_out,
                                   t_first=self.input_tf, intensities=False, workspace=self.workspace, stream=stream)
            else:
                spk_encode_latency(self.image, self.bank, self.T, self.filter_threshold, wave=False, t_first=False,
                                   intensities=self.inten, workspace=self.workspace, stream=stream)
                spk_local_normalization(self.inten, self.local_norm[0], self.local_norm[1], out=self.inten_norm,
                                        stream=stream)
                spk_rank_latency(self.inten_norm, self.T, wave=wave_out, t_first=self.input_tf,
                                 workspace=self.workspace, stream=stream)
            mark("encode", 1)
        x, x_tf = self.input_wave, self.input_tf
        x_exact = x_tf is not None  # x is Eq.1 of x_tf
        last_conv = None
        pooled_by = None  # a pool stage already done by the fused launch of the conv stage before it
        for i, (st, b) in enumerate(zip(self.stages, self.bufs)):
            self._wait_pending(i, main)
            self.pre_waves[i] = x
            self.pre_tf[i] = x_tf if x_exact else None
            if pooled_by is not None:
                x, x_tf, x_exact, pooled_by = b["out"], b["out_tf"], True, None
                continue
            if _is_conv(st):
                mark(f"conv{i}", 0)
                outs = dict(potentials=b["P"], spikes=b["S"], t_first=b["tf"], v_first=b["vf"],
                            workspace=self.workspace, stream=stream)
                s = _stride(st)
                nxt = self.stages[i + 1] if i + 1 < len(self.stages) else None
                if self._fusable(i, x_exact):
                    nb = self.bufs[i + 1]
                    spk_conv_fire_pool(x_tf, self.T, b["weight"], st.pad, st.thr, nxt.P, pooled_t_first=nb["out_tf"],
                                       pooled_wave=nb["out"] if self.want_waves else False, **outs)
                    pooled_by = i
                elif x_exact and s == 1:
                    spk_conv_fire_first_spike(x_tf, self.T, b["weight"], st.pad, st.thr, **outs)
                elif x_exact:
                    spk_conv_fire_first_spike_strided(x_tf, self.T, b["weight"], s, st.pad, st.thr, **outs)
                elif s == 1:
                    spk_conv_fire(x, b["weight"], st.pad, st.thr, **outs)
                else:
                    spk_conv_fire_strided(x, b["weight"], s, st.pad, st.thr, **outs)
                mark(f"conv{i}", 1)
                if early_learn and i in self._side_kwta:
                    side = self._side[self._side_kwta[i]]
                    self._conv_done[i].record(main)
                    side.wait_event(self._conv_done[i])
                    with torch.cuda.stream(side):  # (a hook's events go on the side stream)
                        mark(f"kwta{i}", 0)
                        spk_kwta(b["tf"], b["vf"], self.T, st.k, st.r, winners=b["win"], n_winners=b["nw"],
                                 workspace=b["ws_kwta"], stream=side)
                        mark(f"kwta{i}", 1)
                else:
                    mark(f"kwta{i}", 0)
                    spk_kwta(b["tf"], b["vf"], self.T, st.k, st.r, winners=b["win"], n_winners=b["nw"],
                             workspace=self.workspace, stream=stream)
                    mark(f"kwta{i}", 1)
                if early_learn and i == self._early_at:
                    self._launch_learners(lambda ii: ii <= i, self._forks[0], stream)
                x, x_tf, x_exact = b["S"], b["tf"], False
                last_conv = i
            else:
                mark(f"pool{i}", 0)
                if self.pool_from_first_spike and x_tf is not None:
                    spk_pool_first_spike(x_tf, self.T, st.P, st.R, st.D, out_wave=b["out"] if self.want_waves else False,
                                         out_t_first=b["out_tf"], stream=stream)
                    x_exact = True  # the pooled wave is written as Eq.1 of the pooled map
                else:
                    spk_pool(x, st.P, st.R, st.D, out_wave=b["out"], out_t_first=b["out_tf"], stream=stream)
                    # (pooling an Eq.1 wave gives the Eq.1 wave of the pooled map)
                mark(f"pool{i}", 1)
                x, x_tf = b["out"], b["out_tf"]
        if last_conv is not None and self.stages[last_conv].learn == "rstdp":
            b = self.bufs[last_conv]
            mark("decide", 0)
            spk_decide(b["win"], b["nw"], self.labels, self.n_classes, decision=self.decision, reward=self.reward,
                       stream=stream)
            mark("decide", 1)

    def _fusable(self, i, x_exact):
        """Conv stage i and the pool stage after it run as one spk_conv_fire_pool launch."""
        st = self.stages[i]
        nxt = self.stages[i + 1] if i + 1 < len(self.stages) else None
        if not (self.fused and x_exact and _is_conv(st) and nxt is not None and not _is_conv(nxt)):
            return False
        ho, wo = self.bufs[i]["tf"].shape[2:]
        return (_stride(st) == 1 and not math.isinf(st.thr) and nxt.P == nxt.R and nxt.D == 0 and nxt.P <= min(ho, wo)
                and nxt.P * wo <= 128)

    def _learners(self):
        return [(i, st, b) for i, (st, b) in enumerate(zip(self.stages, self.bufs))
                if _is_conv(st) and st.learn is not None]

    def _apply(self, i, st, b, s):
        common = (self.pre_waves[i], b["win"], b["nw"])
        rates = (st.a_plus, st.a_minus, st.lb, st.ub, st.stabilizer)
        kw = dict(workspace=b["ws_learn"], stream=s)
        stride = _stride(st)
        if not self.want_waves and self.pre_tf[i] is not None and stride == 1:
            # the layer input is kept as its first-spike map only
            if st.learn == "rstdp":
                spk_rstdp_first_spike(b["weight"], st.pad, self.pre_tf[i], self.T, b["win"], b["nw"], self.reward,
                                      *rates, **kw)
            else:
                spk_stdp_first_spike(b["weight"], st.pad, self.pre_tf[i], self.T, b["win"], b["nw"], *rates, **kw)
        elif st.learn == "rstdp" and stride == 1:
            spk_rstdp(b["weight"], st.pad, *common, self.reward, *rates, **kw)
        elif st.learn == "rstdp":
            spk_rstdp_strided(b["weight"], stride, st.pad, *common, self.reward, *rates, **kw)
        elif stride == 1:
            spk_stdp(b["weight"], st.pad, *common, *rates, **kw)
        else:
            spk_stdp_strided(b["weight"], stride, st.pad, *common, *rates, **kw)

    def _launch_learners(self, which, fork, stream):
        """Enqueue, each on its side stream forked from the caller's stream at
        this point, the plasticity of the not yet launched learners i with which(i)."""
        main = stream if stream is not None else torch.cuda.current_stream()
        fork.record(main)
        for j, (i, st, b) in enumerate(self._learners()):
            if i in self._launched or not which(i):
                continue
            s = self._side[j]
            s.wait_event(fork)
            self._apply(i, st, b, s)
            self._joins[j].record(s)
            self._launched.add(i)

    def _wait_pending(self, stage, main):
        """Make `main` wait for the deferred learners of conv stages <= stage + 1
        (stage i writes the input of conv stage i + 1; -1 stands for the source)."""
        for i in [i for i in self._pending if i - 1 <= stage]:
            main.wait_event(self._joins[self._pending.pop(i)])

    def finish(self, stream=None):
        """Join any plasticity left running by step(defer_learn=True) into the stream."""
        main = stream if stream is not None else torch.cuda.current_stream()
        self._wait_pending(len(self.stages), main)

    def learn(self, stream=None, hook=None):
        """Enqueue the plasticity of every learning conv stage not yet started by
        forward(early_learn=True) (names "stdp<i>", or one "learn" span -- the
        part not hidden behind the forward -- when the layers run concurrently)."""
        mark = hook or (lambda name, phase: None)
        main = stream if stream is not None else torch.cuda.current_stream()
        if self.concurrent_learn:
            mark("learn", 0)
            self._launch_learners(lambda i: True, self._forks[1], stream)
            for j in range(len(self._learners())):
                main.wait_event(self._joins[j])
            self._launched.clear()
            mark("learn", 1)
            return
        for i, st, b in self._learners():
            mark(f"stdp{i}", 0)
            self._apply(i, st, b, main)
            mark(f"stdp{i}", 1)

    def step(self, stream=None, hook=None, defer_learn=False):
        """One pass of the whole hot path over the batch: forward, then plasticity
        (the earlier layers' plasticity overlaps the end of the forward).  With
        defer_learn (and concurrent learning) the plasticity is not joined at the
        end of the step: the next forward waits for each layer's update right
        before the stage that rewrites that layer's input (and so before the
        layer's conv), so the last layer's update overlaps the next batch's first
        layers; call finish() (or synchronize the device) before reading weights.
        The results are those of joined steps."""
        self.forward(stream, hook, early_learn=self.concurrent_learn)
        if not (defer_learn and self.concurrent_learn):
            self.learn(stream, hook)
            return
        self._launch_learners(lambda i: True, self._forks[1], stream)
        for j, (i, st, b) in enumerate(self._learners()):
            self._pending[i] = j
        self._launched.clear()


def chain_for(workload, filter_bank=None, device="cuda", **kw):
    """A Chain for a workload description (stages, sizes, source); filter_bank
    is the [C,KF,KF] float tensor of an image source."""
    bank = filter_bank
    if bank is not None and not isinstance(bank, torch.Tensor):
        bank = torch.from_numpy(bank)
    return Chain(workload.stages, workload.B, workload.T, workload.H, workload.W, workload.cin,
                 source=workload.source, filter_bank=bank, n_classes=workload.n_classes, device=device, **kw)


INF = math.inf


class OnlineTrainer:
    """Online plasticity: one image per step, each image's forward run with the
    weights left by the images before it (the tutorial's training loop,
    section "Tutorial", "Training and Testing": each sample goes through the
    network in train mode and its layer's STDP object updates the weights
    before the next sample).  Equal to a sequence of one-image Chain steps.

    A one-image Chain (one stream, compact inter-layer form: no per-step
    potentials) does the work.  With use_graph, `steps_per_graph` consecutive
    steps -- each copying its image and label from a staging slot into the
    chain's inputs, then the chain's forward and plasticity -- are captured
    once in a HIP graph, so steps_per_graph images cost one staging copy and
    one graph launch, with no host work in between.  A trailing partial group
    runs eagerly.  Weights change in place (chain.weights())."""

    def __init__(self, stages, T, H, W, cin, filter_bank, filter_threshold=0.0, n_classes=10, device="cuda",
                 use_graph=True, steps_per_graph=16):
        self.chain = Chain(stages, 1, T, H, W, cin, source="image", filter_bank=filter_bank,
                           filter_threshold=filter_threshold, n_classes=n_classes, device=device,
                           want_potentials=False, want_spikes=False, concurrent_learn=False)
        dev = self.chain.image.device
        self.use_graph = use_graph
        self.K = max(1, int(steps_per_graph))
        self.img_stage = torch.zeros((self.K, H, W), dtype=torch.uint8, device=dev)
        self.lab_stage = torch.zeros((self.K,), dtype=torch.int32, device=dev)
        self.graph = None

    def set_weights(self, weights):
        self.chain.set_weights(weights)

    def set_rates(self, layer, a_plus, a_minus):
        """Rates of conv layer `layer` for the images run from now on; a captured
        graph holds the old rates as kernel arguments, so it is captured again."""
        self.chain.set_rates(layer, a_plus, a_minus)
        self.graph = None

    def weights(self):
        return self.chain.weights()

    def _step_from(self, j):
        self.chain.image.copy_(self.img_stage[j:j + 1])
        self.chain.labels.copy_(self.lab_stage[j:j + 1])
        self.chain.step()

    def _capture(self):
        # one eager step on a side stream first (first launches load the kernels),
        # with the weights it changes restored afterwards
        saved = [w.clone() for w in self.chain.weights()]
        side = torch.cuda.Stream(device=self.chain.image.device)
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            self._step_from(0)
        torch.cuda.current_stream().wait_stream(side)
        for w, v in zip(self.chain.weights(), saved):
            w.copy_(v)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for j in range(self.K):
                self._step_from(j)
        self.graph = g

    def run(self, images, labels=None):
        """Learn from images (u8 [N, H, W] on the device) in order; labels
        (i32 [N]) feed the decision of a reward-modulated last layer."""
        N = images.shape[0]
        i = 0
        while i < N:
            n = min(self.K, N - i)
            self.img_stage[:n].copy_(images[i:i + n])
            if labels is not None:
                self.lab_stage[:n].copy_(labels[i:i + n])
            if self.use_graph and n == self.K:
                if self.graph is None:
                    self._capture()
                self.graph.replay()
            else:
                for j in range(n):
                    self._step_from(j)
            i += n


def online_for(workload, filter_bank, device="cuda", **kw):
    """An OnlineTrainer for a workload description with an image source."""
    bank = filter_bank
    if bank is not None and not isinstance(bank, torch.Tensor):
        bank = torch.from_numpy(bank)
    return OnlineTrainer(workload.stages, workload.T, workload.H, workload.W, workload.cin, bank,
                         n_classes=workload.n_classes, device=device, **kw)
