"""Batch-size nomenclature of Appendix A (the list after Algorithm 1 and the Option 1 /
Option 2 table): how the learner's batch quantities follow from world_size,
local_num_envs, num_steps, num_minibatches and update_epochs."""
from __future__ import annotations


def derive(world_size, local_num_envs, num_steps, num_minibatches, update_epochs=1):
    """Return the derived hyperparameters as a dict.

    num_envs = world_size * local_num_envs
    local_batch_size = local_num_envs * num_steps;  batch_size = world_size * local_batch_size
    local_minibatch_size = local_batch_size / num_minibatches
    minibatch_size = world_size * local_minibatch_size
    gradient updates per learning phase = update_epochs * num_minibatches
    """
    local_batch = local_num_envs * num_steps
    if local_batch % num_minibatches:
        raise ValueError("local_batch_size must split evenly into num_minibatches")
    local_mb = local_batch // num_minibatches
    return dict(world_size=world_size, local_num_envs=local_num_envs,
                num_envs=world_size * local_num_envs, num_steps=num_steps,
                local_batch_size=local_batch, batch_size=world_size * local_batch,
                num_minibatches=num_minibatches, local_minibatch_size=local_mb,
                minibatch_size=world_size * local_mb,
                updates=update_epochs * num_minibatches)
