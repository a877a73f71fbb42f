"""A tiny Llama-shaped model (untied embedding and LM head, GQA-like k, SwiGLU-shaped FFN, RMSNorm
weights), shared by the optimizer test on the GPU and the CPU emulation test of its gradients."""
import torch


class Block(torch.nn.Module):
    def __init__(self, d, kv, f):
        super().__init__()
        self.q = torch.nn.Linear(d, d, bias=False)
        self.k = torch.nn.Linear(d, kv, bias=False)
        self.o = torch.nn.Linear(kv, d, bias=False)
        self.gate = torch.nn.Linear(d, f, bias=False)
        self.down = torch.nn.Linear(f, d, bias=False)
        self.norm = torch.nn.Parameter(torch.ones(d))

    def forward(self, x):
        h = x * self.norm
        x = x + self.o(torch.tanh(self.k(h))) + self.q(h)
        return x + self.down(torch.nn.functional.silu(self.gate(x)))


class Tiny(torch.nn.Module):
    def __init__(self, vocab=96, d=64, kv=32, f=160):
        super().__init__()
        self.embed = torch.nn.Embedding(vocab, d)
        self.blocks = torch.nn.ModuleList([Block(d, kv, f) for _ in range(2)])
        self.final_norm = torch.nn.Parameter(torch.ones(d))
        self.lm_head = torch.nn.Linear(d, vocab, bias=False)

    def forward(self, tok):
        x = self.embed(tok)
        for b in self.blocks:
            x = b(x)
        return self.lm_head(x * self.final_norm)


def tiny_bf16_gradients(seed: int, device: str = "cpu"):
    """A bf16 Tiny model after one backward pass on 4 x 24 random tokens (92 predicted positions)."""
    torch.manual_seed(seed)
    model = Tiny().to(device).to(torch.bfloat16)
    tok = torch.randint(0, 96, (4, 24), device=device)
    loss = torch.nn.functional.cross_entropy(model(tok[:, :-1]).float().reshape(-1, 96), tok[:, 1:].reshape(-1))
    loss.backward()
    return model
