"""CPU oracle for the batched speculative-decoding step (test infrastructure).

This package is test infrastructure only.  It is imported by the tests, by the
smoke check and by the benchmark's CPU-baseline leg, never by the GPU path,
and it shares no code with it: it is plain numpy in float64, written from the
paper's statement of the method.

What it computes, and where the paper states it:

* ``model``  -- the target forward.  Verification runs one target forward over
  the committed context plus the draft block and reads the target
  distribution at every block position (Sec. 3.1, Eq. verification-context;
  App. "Draft-Path Reconstruction": verification is one forward over the
  draft path).  The decoder is the standard pre-norm RMSNorm / RoPE / GQA /
  SwiGLU layer of the backbones the paper uses (App. "Models and Draft
  Heads").  Pinned by its plain definition (a causal forward over the whole
  sequence without a cache) and by closed-form special cases.
* ``accept`` -- the accept rule of Sec. 2.2 (Eq. accept-rule), the residual
  resample at the first rejection and the bonus token, plus greedy prefix
  matching.  Pinned by the four checks of the method (draft length 0 is
  autoregressive decoding, a draft equal to the greedy choice is fully
  accepted, greedy acceptance is the longest argmax-matching prefix, and the
  committed tokens are distributed as the target), by Eq. alpha and by brute
  force on tiny vocabularies.  The top-p variant of the paper's evaluation
  setting (both distributions truncated to their nucleus) is pinned by the
  same distribution check on the nucleus of the target, by its reduction to
  greedy decoding as top_p goes to 0 and by hand-worked nuclei.
* ``record`` -- the cycle record's verification distributions: the target's
  top-64 log-probabilities per draft position, full-vocabulary normalised,
  in bf16 (App. "Implementing Draft-Path Reconstruction in verl").  Pinned by
  brute force (a full sort and an independent log-sum-exp) on small rows.
* ``dca``    -- the depth-coupled acceptance loss with verify-gated masking over
  the record's top-64 support plus one residual bin, and its gradient with
  respect to the head logits (Sec. "The Depth-Coupled Acceptance Loss",
  "Learning up to the First Rejection"; App. "DCA").  Pinned by float64
  autograd of an independent torch form, by Eq. alpha's identity alpha = 1 - TV
  when the record covers the vocabulary, by Eq. dca-identity, by the range of
  Eq. dca-tail and by the closed forms of VGM.
* ``kv``     -- commit/rollback of the KV index (Sec. 2.2; App. "Train--Inference
  Inconsistency under Teacher Forcing", Eq. tf-restart-kv).  Closed form.
* ``mtp``    -- the recurrent MTP draft head (Sec. 2.2; App. "Models and Draft
  Heads"; Eqs. tf-restart and tf-restart-kv), and the draft-path
  reconstruction that re-runs recorded chains with the recorded drafts as
  inputs (App. "Draft-Path Reconstruction").  Pinned by pass-through special
  cases (concat order, shared embedding and head, final norm, the chain's
  feed), by two special cases in which the decoder layer has a closed form that
  reads the head's cache (uniform attention; scores fixed by RoPE's
  relative-position property), which fix the (hidden, token) pair and the
  rotary position of every extend and chain entry, and by the reconstruction
  reproducing the drafting's own distributions.
* ``mixing`` -- the draft construction of the top-1 mixing workloads (an input
  recipe, not part of the method).

Precision: float64 throughout.  ``Rounding("contract")`` rounds to bfloat16
exactly the tensors that the bf16 GPU path feeds to its matrix cores (the
rounding contract), so that integer decisions can be compared bit for bit.
"""
from .numerics import Rounding, round_bf16, softmax, rmsnorm, silu, rope, inverse_cdf, inverse_cdf_rows, nucleus  # noqa: F401
from .model import attention, layer_forward, verify_forward, full_forward, prefill, ar_decode  # noqa: F401
from .accept import spec_accept, AcceptResult  # noqa: F401
from .record import record_topk  # noqa: F401
from .dca import dca_loss  # noqa: F401
from .kv import kv_commit  # noqa: F401
from .mtp import mtp_apply, mtp_draft, mtp_reconstruct  # noqa: F401
from .mixing import mixing_drafts  # noqa: F401
