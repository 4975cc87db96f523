"""torch.autograd wrapper: the fused kernels produce the gradient in the forward
call; backward only scales it by the upstream gradient of the (reduced) loss."""
import torch

from .binding import rnnt_loss


class _RNNTLossFunction(torch.autograd.Function):
    @staticmethod
    def forward(ctx, logits, labels, logit_lens, label_lens, blank, variant, reduction):
        loss, grad = rnnt_loss(logits, labels, logit_lens, label_lens, blank=blank, variant=variant,
                               need_grad=logits.requires_grad)
        ctx.reduction = reduction
        ctx.batch = loss.shape[0]
        ctx.save_for_backward(grad if grad is not None else torch.empty(0))
        if reduction == "sum":
            return loss.sum()
        if reduction == "mean":
            return loss.mean()
        return loss

    @staticmethod
    def backward(ctx, grad_loss):
        (grad,) = ctx.saved_tensors
        if ctx.reduction == "none":
            scale = grad_loss.to(torch.float32).view(-1, 1, 1, 1)
        elif ctx.reduction == "mean":
            scale = grad_loss.to(torch.float32) / ctx.batch
        else:
            scale = grad_loss.to(torch.float32)
        g = (grad.to(torch.float32) * scale).to(grad.dtype)
        return g, None, None, None, None, None, None


def rnnt_loss_autograd(logits, labels, logit_lens, label_lens, blank=0, variant="rnnt", reduction="mean"):
    """Differentiable RNN-T / W-RNNT loss; reduction in {"none", "sum", "mean"}."""
    if reduction not in ("none", "sum", "mean"):
        raise ValueError("reduction must be none, sum or mean")
    return _RNNTLossFunction.apply(logits, labels, logit_lens, label_lens, blank, variant, reduction)


class RNNTLoss(torch.nn.Module):
    def __init__(self, blank=0, variant="rnnt", reduction="mean"):
        super().__init__()
        self.blank, self.variant, self.reduction = blank, variant, reduction

    def forward(self, logits, labels, logit_lens, label_lens):
        return rnnt_loss_autograd(logits, labels, logit_lens, label_lens, self.blank, self.variant, self.reduction)
